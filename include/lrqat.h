/*
 * lrqat.h -- C ABI of the LR-QAT linear layer for AMD MI355X (gfx950).
 *
 * LR-QAT (Bondarenko et al., "Low-Rank Quantization-Aware Training for LLMs",
 * arXiv 2406.06385) trains a quantised linear layer through low-rank
 * auxiliary matrices placed inside the rounding operator (Section 3,
 * Eq. lr_qat):
 *
 *     W_hat = s * clip( round( Phi0 + (alpha/r) * A * B ), -2^(b-1), 2^(b-1)-1 )
 *
 * with W0 in R^{m x k} (m = out features, k = in features, as nn.Linear),
 * the frozen downcast Phi0 = phi(W0 / s0) (Section 3, Eq. phi), trainable
 * A in R^{m x r}, B in R^{r x k} and scale s.  Tokens are rows:
 * Y = X * W_hat^T with X in R^{T x k}.  Gradients use the straight-through
 * estimator for round() (Section 3, 'QAT with low-rank adapters') and W_hat
 * is recomputed in the backward pass instead of being kept from the forward
 * (Section 3, 'Gradient checkpointing').
 *
 * Conventions shared by every entry point
 *   - Tensor arguments are DEVICE pointers, dense row-major, owned by the
 *     caller; the library keeps no pointer after a call returns.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream).  Results are visible after the stream is synchronised.
 *   - The library allocates no device memory at run time.  Scratch space comes
 *     from the caller as a workspace sized by the *_workspace_size queries
 *     (lrqat_backward_static alone uses an array the library holds on each
 *     GPU).
 *   - Every argument is validated on the host before any HIP call; invalid
 *     arguments return an error status and launch nothing.  A failed launch
 *     returns LRQAT_EHIP.  No C++ exception crosses this interface.
 *     lrqat_last_error() gives a message for the last failure of the
 *     calling thread.
 *   - Calls that share a workspace must not overlap in time.
 *   - Pointers to tensors read as 16-byte vectors must be 16-byte aligned
 *     (X, Y, dY, dX, Phi0, W_int4, the workspace); A, B, s, z, dA, dB, ds and
 *     W0 must be 4-byte aligned.
 */
#ifndef LRQAT_H
#define LRQAT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LRQAT_OK = 0,
  LRQAT_EINVAL = 1,        /* a null pointer, a size out of range, misalignment */
  LRQAT_EUNSUPPORTED = 2,  /* a valid combination this library does not run */
  LRQAT_EWORKSPACE = 3,    /* workspace smaller than the size query returns */
  LRQAT_EHIP = 4           /* a HIP runtime or launch error */
} lrqat_status;

/* Storage format of Phi0 (Section 3, 'Downcasting operator'). */
typedef enum {
  /* Fixed point Qb.(8-b) in int8 (Eq. phi_fixed_point): int8 [m][k], value
   * code / 2^(8-b).  2 <= b <= 7. */
  LRQAT_PHI_FIXED_Q8 = 0,
  /* INT-b, two per byte ("double-packed"): uint8 [m][k/2]; byte j of a row
   * holds column 2j in its low nibble and column 2j+1 in its high nibble, as
   * 4-bit two's complement.  2 <= b <= 4, k even. */
  LRQAT_PHI_INT_PACKED2 = 1
} lrqat_phi_format;

/* Element type of the activations X, Y, dY, dX ("compute data type",
 * Section 4.2).  A, B, s, s0, W0, dA, dB, ds are always float32. */
typedef enum { LRQAT_FP32 = 0, LRQAT_BF16 = 1 } lrqat_dtype;

typedef struct {
  int64_t out_features;  /* m >= 1 */
  int64_t in_features;   /* k >= 1 */
  int32_t rank;          /* r, 1 <= r <= 256 */
  float alpha;           /* the factor alpha of alpha/r (finite) */
  int32_t bits;          /* b, see lrqat_phi_format */
  int32_t phi_format;    /* lrqat_phi_format */
  int64_t group_size;    /* 0: one scale per output channel, s[m];
                            g > 0: one scale per row and group of g consecutive
                            input columns, s[m][k/g] (Section 4, 'g128');
                            k % g == 0 and g % 32 == 0 */
  int32_t act_bits;      /* 0: X used as is; 8: per-token dynamic symmetric
                            int8 fake quantisation of X with s_x[t] =
                            max|X[t,:]|/127 and a straight-through gradient
                            (Section 4, weight-activation quantisation);
                            needs act_dtype = LRQAT_BF16 */
  int32_t act_dtype;     /* lrqat_dtype */
} lrqat_layer;

/* Bytes of workspace lrqat_forward / lrqat_backward need for `tokens` rows.
 * Returns 0 for an invalid layer (see lrqat_last_error()). */
size_t lrqat_forward_workspace_size(const lrqat_layer* layer, int64_t tokens);
size_t lrqat_backward_workspace_size(const lrqat_layer* layer, int64_t tokens);

/*
 * Setup: range estimation and downcast (Section 3, Eq. phi).
 * From the pretrained weight W0 (float32 [m][k]) compute the initial scale
 * by min-max range estimation, s0 = max|W0 over a row or row-group| /
 * (2^(b-1)-1) (an all-zero row or group gets s0 = 1), and the frozen
 * Phi0 = phi(W0 / s0) in `layer->phi_format`: fixed point
 * INT8(round(2^(8-b) clip(W0/s0))) (Eq. phi_fixed_point) or double-packed
 * INT-b clip(round(W0/s0)).  round() is half-to-even; the quotient and the
 * rounding decision are float32.  s0_out: float32 [m] or [m][k/g];
 * phi0_out: int8 [m][k] or uint8 [m][k/2].
 *
 * Asymmetric quantisation (Eq. dequant; the zero offset z is set at range
 * estimation and frozen, Section 4): with z0_out (int32, shaped like s0) the
 * range [min(W0, 0), max(W0, 0)] of a row or group maps onto the grid:
 * s0 = (max - min) / (2^b - 1), z0 = clip(-2^(b-1) - round(min / s0)), and
 * Phi0 carries the offset, z0 added outside the rounding of the downcast:
 * fixed point clip(round(2^(8-b) W0/s0) + 2^(8-b) z0), INT-b
 * clip(round(W0/s0) + z0).  z0_out = NULL: symmetric.
 */
lrqat_status lrqat_init_from_weights(const lrqat_layer* layer, const float* W0,
                                     float* s0_out, int32_t* z0_out, void* phi0_out, void* stream);

/*
 * Setup with L^p-norm range estimation (Section 4 'Baselines', Appendix B
 * 'PTQ initialization': the range minimising the L^p norm between quantized
 * and unquantized weights, p in {2, 2.4, 3, 3.5, 4, 5} in the paper).  For
 * each row (or row-group) the candidates are the clipping ratios j / n_grid,
 * j = 1..n_grid, of the min-max range, s_j = (j / n_grid) max|W0| /
 * (2^(b-1)-1) in float32, with error E_j = sum |W0 - s_j clip(round(W0 /
 * s_j))|^p (float32 terms, float64 sums); the smallest j of the minimal E_j
 * gives s0.  Then Phi0 = phi(W0 / s0) as in lrqat_init_from_weights.
 * 1 <= p <= 16, 1 <= n_grid <= 10000; a row or group holds at most 16384
 * weights.
 */
lrqat_status lrqat_init_lp(const lrqat_layer* layer, const float* W0, float p, int n_grid,
                           float* s0_out, void* phi0_out, void* stream);

/*
 * LoftQ initialisation with one alternating step (Section 3 'Downcasting
 * operator', Section 4.2 ablation): for INT-b Phi0 (phi_format
 * LRQAT_PHI_INT_PACKED2) from W0 and a given scale s0 (min-max or L^p), with
 * x = W0 / s0: Phi0 = clip(round(x)), and A [m][r], B [r][k] whose product
 * (alpha/r) A B approximates the dropped fractional part R = x - Phi0 by
 * its best rank-r approximation, split evenly (A^T A = B B^T).  The
 * approximation comes from randomized subspace iteration (r + 16 columns,
 * n_iter iterations, CholeskyQR2 orthonormalisation, Jacobi on the small
 * Gram matrix; 32 iterations capture over 99.9% of the optimal rank-r energy
 * of a noise-like R).  sigma_out (nullable): the r singular values found.
 * rank <= 48, alpha / r > 0.  ws: lrqat_init_loftq_workspace_size() bytes
 * (R in float32 plus the subspace blocks).
 */
size_t lrqat_init_loftq_workspace_size(const lrqat_layer* layer);
lrqat_status lrqat_init_loftq(const lrqat_layer* layer, const float* W0, const float* s0, int n_iter,
                              void* phi0_out, float* A_out, float* B_out, float* sigma_out, void* ws,
                              size_t ws_bytes, void* stream);

/*
 * Forward pass (Section 3, Eq. lr_qat): Y = X_hat * W_hat^T.
 *   X     [T][k] act_dtype     layer input (X_hat = X, or its int8 fake
 *                               quantisation when act_bits = 8)
 *   phi0  Phi0 in phi_format   frozen downcast weight
 *   s     float32 [m] or [m][k/g]
 *   z     int32, shaped like s: the integer zero offset of asymmetric
 *         quantisation (Eq. dequant; Section 3 last paragraph: z outside the
 *         rounding), W_hat = s * (clip(round(Phi0 + (alpha/r) A B)) - z), with
 *         Phi0 already carrying the offset (lrqat_init_from_weights);
 *         NULL for symmetric quantisation
 *   A     float32 [m][r],  B float32 [r][k]
 *   Y     [T][m] act_dtype     output, overwritten
 *   ws    workspace of at least lrqat_forward_workspace_size() bytes
 * Nothing is saved for the backward pass.  T = 0 is a no-op.
 */
lrqat_status lrqat_forward(const lrqat_layer* layer, int64_t tokens, const void* X,
                           const void* phi0, const float* s, const int32_t* z, const float* A,
                           const float* B, void* Y, void* ws, size_t ws_bytes, void* stream);

/*
 * Backward pass with the straight-through estimator (Section 3).  W_hat and
 * its clip mask are recomputed from (Phi0, A, B, s); then
 *   dX = dY * W_hat                             [T][k] act_dtype (nullable:
 *                                               skipped when NULL)
 *   dW = dY^T * X_hat,  G = s (.) M (.) dW       (never written to memory)
 *   dA = (alpha/r) G B^T                        float32 [m][r]
 *   dB = (alpha/r) A^T G                        float32 [r][k]
 *   ds = sum over a row (or row-group) of       float32, shaped like s
 *        dW (.) (q - z)                         (nullable: skipped when NULL;
 *                                               the STE gradient of the
 *                                               learned scale, Section 3)
 * M is the clip mask [lo <= round(Phi0 + (alpha/r) A B) <= hi] and
 * q = clip(round(Phi0 + (alpha/r) A B)) the integer grid (z = 0 when NULL).
 * accumulate = 0 overwrites dA, dB (and ds); 1 adds into them (gradient
 * accumulation over micro-batches).  With T = 0 they are zeroed
 * (accumulate = 0) or left unchanged.  dA, dB and ds are deterministic: the
 * same inputs give the same bits.
 */
lrqat_status lrqat_backward(const lrqat_layer* layer, int64_t tokens, const void* X,
                            const void* phi0, const float* s, const int32_t* z, const float* A,
                            const float* B, const void* dY, void* dX, float* dA, float* dB,
                            float* ds, int accumulate, void* ws, size_t ws_bytes, void* stream);

/*
 * lrqat_backward without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving or
 * training loops, harnesses that forbid hipMalloc).  Same arguments, results
 * and errors as lrqat_backward; the scratch space is one array in device
 * memory that the library holds on each GPU it runs on until the process
 * ends, of lrqat_backward_static_capacity() bytes (64 MiB: enough for a
 * 4096 x 4096 layer with 8192 tokens).  A layer whose
 * lrqat_backward_workspace_size() exceeds it is rejected with
 * LRQAT_EWORKSPACE before anything is launched.  The call allocates nothing.
 * Every call on one GPU uses that GPU's array: calls that overlap in time on
 * one GPU (on different streams or threads) race and must be serialised by
 * the caller.  Nothing in the array has to start at any particular value.
 */
lrqat_status lrqat_backward_static(const lrqat_layer* layer, int64_t tokens, const void* X,
                                   const void* phi0, const float* s, const int32_t* z,
                                   const float* A, const float* B, const void* dY, void* dX,
                                   float* dA, float* dB, float* ds, int accumulate, void* stream);

/* Bytes of the device array lrqat_backward_static uses on each GPU. */
size_t lrqat_backward_static_capacity(void);

/*
 * Merge for inference (Section 3: the adapters fuse into one b-bit integer
 * matrix without loss): W_Z = clip(round(Phi0 + (alpha/r) A B)), written
 * double-packed as uint8 [m][k/2] in the nibble order of
 * LRQAT_PHI_INT_PACKED2; the inference weight is s (.) (W_Z - z).  Needs
 * b <= 4 and k even.  No workspace.
 */
lrqat_status lrqat_merge_to_int4(const lrqat_layer* layer, const void* phi0, const float* A,
                                 const float* B, uint8_t* W_int4, void* stream);

/*
 * Inference on the merged weights (Section 3: after training W_hat = s W_Z,
 * "without any extra overhead"): Y = X_hat (s (.) (W_Z - z))^T, with W_Z the
 * packed int4 output of lrqat_merge_to_int4 (layer->bits <= 4; phi_format is
 * not used), X_hat = X or its per-token int8 fake quantisation when
 * act_bits = 8 (W4A8), s float32 and z int32 (nullable) shaped like the
 * layer's scale.  The same GEMM as lrqat_forward without the grid pass.
 * ws: at least lrqat_infer_workspace_size() bytes (activation codes under
 * W4A8; a re-laid copy of W_Z when k is not a multiple of 32).
 */
size_t lrqat_infer_workspace_size(const lrqat_layer* layer, int64_t tokens);
lrqat_status lrqat_infer_forward(const lrqat_layer* layer, int64_t tokens, const void* X,
                                 const uint8_t* W_int4, const float* s, const int32_t* z, void* Y,
                                 void* ws, size_t ws_bytes, void* stream);

/*
 * Optimizer step for the trainable tensors (Appendix B, Table B1): AdamW with
 * decoupled weight decay (p <- p (1 - lr wd); m <- b1 m + (1 - b1) g;
 * v <- b2 v + (1 - b2) g^2; p <- p - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)),
 * on gradients clipped together to an L2 norm of at most max_grad_norm
 * (g <- g min(1, max_grad_norm / (||g||_2 + 1e-6)), the norm taken over all
 * groups of the call; max_grad_norm <= 0 disables clipping), with the
 * learning rate of step t (1-based) lr_max * (t-1)/W during the first W =
 * warmup_steps steps and lr_max * (N - (t-1)) / (N - W) after them, never
 * below zero (N = total_steps).  The paper's setting: betas (0.9, 0.95),
 * weight decay 0, clipping at 1.0, W = N / 10, separate maximum learning
 * rates for A, B and for s.
 * Each group is a contiguous float32 range of n elements (param, grad and
 * the two moment buffers, all device pointers; moments start at zero) with
 * its own lr_max and weight_decay; at most 32 groups per call (keep a
 * model's adapters in one buffer).  grad_norm_out (device float, nullable)
 * receives the norm before clipping.  Deterministic.  ws: at least
 * lrqat_adamw_workspace_size() bytes.
 */
typedef struct {
  float* param;
  const float* grad;
  float* exp_avg;
  float* exp_avg_sq;
  int64_t n;
  float lr_max;
  float weight_decay;
} lrqat_param_group;

typedef struct {
  float beta1, beta2, eps;
  float max_grad_norm;
  int64_t total_steps, warmup_steps;
} lrqat_adamw_config;

size_t lrqat_adamw_workspace_size(int n_groups, const lrqat_param_group* groups);
lrqat_status lrqat_adamw_step(const lrqat_adamw_config* cfg, int64_t step, int n_groups,
                              const lrqat_param_group* groups, float* grad_norm_out, void* ws,
                              size_t ws_bytes, void* stream);

/* Human-readable name of a status code (static string). */
const char* lrqat_status_string(lrqat_status status);

/* Message describing the last failed call on the calling thread ("" if none). */
const char* lrqat_last_error(void);

/*
 * Per-kernel timing, for profiling.  When enabled, every kernel the library
 * launches is bracketed by HIP events on its stream.  lrqat_timing_read()
 * waits for those events and returns, for up to `max_kernels` kernel names,
 * the name, the number of launches and their summed duration in
 * milliseconds since the last reset; it returns the number of entries
 * written (or -1 on a HIP error).  Names point to static strings.
 */
void lrqat_timing_enable(int enable);
void lrqat_timing_reset(void);
int lrqat_timing_read(const char** names, int64_t* launches, double* total_ms, int max_kernels);

#ifdef __cplusplus
}
#endif

#endif /* LRQAT_H */
