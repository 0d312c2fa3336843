// Kernel argument blocks and host-side launchers of the LR-QAT library.
#pragma once

#include "common.h"

namespace lrqat {

// Integer grid pass (reconstruction / merge).
struct GridArgs {
  const uint8_t* phi0;   // Phi0: int8 [m][ld_phi] (fixed point) or uint8 [m][ld_phi] packed
  int64_t ld_phi;        // bytes per row of phi0
  const float* A;        // [m][r]
  const float* B;        // [r][k]
  int64_t m, k;
  int r;
  float c;               // alpha / r
  double c64;            // alpha / r in float64 (for the exact re-decision)
  int bits;
  int packed;            // 1: Phi0 is double-packed INT-b
  uint8_t* qout;         // q [m][ldq]: packed int4, or int8 when q8out
  int64_t ldq;           // bytes per row of qout
  int64_t kq;            // columns written per row of qout (>= k; columns >= k are 0)
  int q8out;             // 1: q as int8 (grids of 5..7 bits)
  uint16_t* mout;        // clip-mask bits: bit (col % 16) of word [row][col / 16] (nullable)
  int64_t ldm;           // 16-bit words per row of mout (kq / 16)
  float tau_coef;        // set by launch_grid: error-bound coefficient of the float32 delta
  int nit;               // set by launch_grid: 16-row rounds per wave
};

// bf16 MFMA GEMM family.  C[M][N] = sum_K a(M, K) b(K, N) with the operand
// sources and epilogue chosen by the kernel variant.
enum GemmVariant { kFwd = 0, kDx = 1, kDw = 2 };

struct GemmArgs {
  int64_t M, N, K;
  const void* a;          // kFwd: X bf16 [T][k] or n int8 [T][lda]; kDx: dY [T][m]; kDw: dY [T][m]
  int64_t lda;
  const void* b;          // kFwd/kDx: q [m][ldb], packed int4 or int8; kDw: X bf16 [T][k] or n int8 [T][ldb]
  int64_t ldb;
  const float* s;         // weight scale [m] or [m][ngroups]
  const int32_t* z;       // zero offset, shaped like s (variants with kOptZ)
  int64_t gsize, ngroups;
  const float* sx;        // per-token activation scale [T] (W4A8) or null
  void* out;              // kFwd: Y [T][m]; kDx: dX [T][k]
  int64_t ldo;
  const uint16_t* mask;   // kDw: clip-mask bits, bit (col % 16) of word [row][col / 16]
  int64_t ldm;            // 16-bit words per row of mask
  const float* Am;        // kDw: A [m][r]
  const float* Bm;        // kDw: B [r][k]
  int r;
  float* dA_part;         // kDw: [ceil(N/256)][M][r]
  float* dB_part;         // kDw: [ceil(M/256)][r][N]
  const uint8_t* qd;      // kDw with kOptDs: q [M][ldqd] (packed int4, or int8 with kOptQ8)
  int64_t ldqd;
  float* ds_part;         // kDw, nullable: [M][ldds], sums over 32-column chunks of dW (q - z)
  int64_t ldds;
  int qd8;                // kDw with ds_part: qd is int8
};

// Variant options of the forward and dX GEMMs (bit flags).
enum : int {
  kOptZ = 1,   // zero offset: the weight operand is s (q - z)
  kOptQ8 = 2   // the integer grid q is int8 (grids of 5..7 bits) instead of packed int4
};

constexpr int GEMM_BM = 256, GEMM_BN = 256, GEMM_BK = 64;

hipError_t launch_minmax_scale(const float* W0, int64_t m, int64_t k, int64_t gsize, int bits, float* s0, int32_t* z0,
                               hipStream_t st);
hipError_t launch_encode(const float* W0, const float* s0, const int32_t* z0, int64_t m, int64_t k, int64_t gsize,
                         int bits, int packed, void* phi0, hipStream_t st);
hipError_t launch_grid(const GridArgs& a, hipStream_t st);
// per-token int8 quantisation of bf16 X [T][k]: codes n [T][ldn] and/or X_hat in bf16 [T][ldh] (nullable), s_x [T]
hipError_t launch_act_quant(const uint16_t* X, int64_t T, int64_t k, int8_t* n, int64_t ldn, uint16_t* xh, int64_t ldh,
                            float* sx, hipStream_t st);
// opt: kOpt* flags (forward and dX; the dW GEMM takes its options at run time)
hipError_t launch_gemm(GemmVariant v, bool act, bool grouped, int opt, const GemmArgs& p, hipStream_t st);
// per-family launchers, one translation unit each for parallel builds
hipError_t launch_fwd_i4(bool grouped, bool zp, const GemmArgs& p, hipStream_t st);      // gemm_fwd.hip
hipError_t launch_fwd_i8(bool grouped, bool zp, const GemmArgs& p, hipStream_t st);      // gemm_fwd_q8.hip
hipError_t launch_fwd_act_i4(bool grouped, bool zp, const GemmArgs& p, hipStream_t st);  // gemm_fwd_act.hip
hipError_t launch_fwd_act_i8(bool grouped, bool zp, const GemmArgs& p, hipStream_t st);  // gemm_fwd_act_q8.hip
hipError_t launch_dx_i4(bool grouped, bool zp, const GemmArgs& p, hipStream_t st);       // gemm_dx.hip
hipError_t launch_dx_i8(bool grouped, bool zp, const GemmArgs& p, hipStream_t st);       // gemm_dx_q8.hip
hipError_t launch_dw_pc(const GemmArgs& p, hipStream_t st);                              // gemm_dw.hip
hipError_t launch_dw_grp(const GemmArgs& p, hipStream_t st);                             // gemm_dw_grp.hip
// rows of w bytes re-laid with a leading dimension of ldd bytes, zero-filled
hipError_t launch_repack_rows(const uint8_t* src, int64_t m, int64_t w, uint8_t* dst, int64_t ldd, hipStream_t st);
// ds[row][grp] = (accumulate ? ds : 0) + sum of the 32-column chunk partials of the group
hipError_t launch_reduce_ds(const float* part, int64_t m, int64_t ldpart, int64_t nchunks, int64_t chunks_per_group,
                            int64_t ngroups, float* ds, int accumulate, hipStream_t st);
hipError_t launch_reduce(const float* part, int64_t nparts, int64_t n, float* out, float c, int accumulate,
                         hipStream_t st);
struct Reduce2Args {        // side 0: dA, side 1: dB
  const float* part[2];     // [nparts][n] partial sums
  int64_t nparts[2], n[2];
  float* out[2];
  int vec[2];               // 16-byte aligned rows and n % 4 == 0
  float c;
  int accumulate;
};
hipError_t launch_reduce2(const Reduce2Args& ra, hipStream_t st);

// float32 activation path (simple tiled FMA kernels).
struct F32Args {
  int64_t T, m, k;
  int r;
  float c;
  const float* X;
  const float* dY;
  const uint8_t* q;       // q [m][ldq], packed int4 or int8 (q8)
  int64_t ldq;
  int q8;
  const uint16_t* mask;   // clip-mask bits, bit (col % 16) of word [row][col / 16]
  int64_t ldm;            // 16-bit words per row
  const float* s;
  const int32_t* z;       // zero offset shaped like s, or null
  int64_t gsize, ngroups;
  const float* A;
  const float* B;
  float* dW;              // workspace [m][k]
};
hipError_t launch_f32_forward(const F32Args& a, float* Y, hipStream_t st);
hipError_t launch_f32_dx(const F32Args& a, float* dX, hipStream_t st);
hipError_t launch_f32_dw(const F32Args& a, float* dA, float* dB, float* ds, int accumulate, hipStream_t st);

// AdamW step with global L2 clipping (optim.hip).
struct OptimGroup {
  float* param;
  const float* grad;
  float* exp_avg;
  float* exp_avg_sq;
  int64_t n;
  float lr_max, weight_decay;
};
constexpr int kMaxOptimGroups = 32;
struct OptimArgs {
  OptimGroup g[kMaxOptimGroups];
  int64_t first[kMaxOptimGroups + 1];  // first chunk of each group (set by optim_prepare)
  int ngroups;
  int64_t step, total, warmup;
  float beta1, beta2, eps, max_norm;
};
void optim_prepare(OptimArgs& a);
int64_t optim_chunks(const OptimArgs& a);
hipError_t launch_adamw(const OptimArgs& a, double* part, float* norm_coef, float* norm_out, hipStream_t st);

}  // namespace lrqat
