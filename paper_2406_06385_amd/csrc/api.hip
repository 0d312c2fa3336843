// Host side of the C ABI declared in include/lrqat.h: argument validation,
// workspace layout and the kernel sequence of each entry point.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "init.h"
#include "kernels.h"
#include "lrqat.h"

using namespace lrqat;

namespace {

thread_local std::string g_last_error;

lrqat_status fail(lrqat_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
lrqat_status fail(lrqat_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

// ------------------------------------------------------------------ kernel timing
struct Pending {
  const char* name;
  hipEvent_t start, stop;
};
std::mutex g_timing_mu;
bool g_timing = false;
std::vector<Pending> g_pending;
struct Totals {
  int64_t launches = 0;
  double ms = 0.0;
};
std::map<std::string, std::pair<const char*, Totals>> g_totals;

template <class F>
hipError_t timed(const char* name, hipStream_t st, F&& launch) {
  bool on;
  {
    std::lock_guard<std::mutex> lk(g_timing_mu);
    on = g_timing;
  }
  if (!on) return launch();
  hipEvent_t a, b;
  if (hipEventCreate(&a) != hipSuccess) return hipErrorOutOfMemory;
  if (hipEventCreate(&b) != hipSuccess) {
    (void)hipEventDestroy(a);
    return hipErrorOutOfMemory;
  }
  (void)hipEventRecord(a, st);
  hipError_t e = launch();
  (void)hipEventRecord(b, st);
  std::lock_guard<std::mutex> lk(g_timing_mu);
  g_pending.push_back({name, a, b});
  return e;
}

// ------------------------------------------------------------------ layout
constexpr int64_t kMaxDim = int64_t(1) << 22;  // keeps 32-bit buffer offsets within a 256-row tile

inline int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }
inline bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

struct Dims {
  int64_t m, k, r, g, ngroups, kpad, mpad;
  int bits, packed, act, bf16;
  int q8w;  // the integer grid is kept as int8 (fixed-point Phi0 with b = 5..7)
  float c;
  double c64;
  bool alpha_nonpos() const { return !(c64 > 0.0); }
};

struct Workspace {
  size_t q = 0, mask = 0, n = 0, xh = 0, sx = 0, dA_part = 0, dB_part = 0, ds_part = 0, dW = 0, total = 0;
};

lrqat_status check_layer(const lrqat_layer* L, Dims& d) {
  if (!L) return fail(LRQAT_EINVAL, "layer is NULL");
  if (L->out_features < 1 || L->in_features < 1 || L->out_features > kMaxDim || L->in_features > kMaxDim)
    return fail(LRQAT_EINVAL, "out_features and in_features must be in [1, 2^22] (got %lld, %lld)",
                (long long)L->out_features, (long long)L->in_features);
  if (L->rank < 1 || L->rank > 256) return fail(LRQAT_EINVAL, "rank must be in [1, 256] (got %d)", L->rank);
  if (!std::isfinite(L->alpha)) return fail(LRQAT_EINVAL, "alpha must be finite");
  if (L->phi_format != LRQAT_PHI_FIXED_Q8 && L->phi_format != LRQAT_PHI_INT_PACKED2)
    return fail(LRQAT_EINVAL, "unknown phi_format %d", L->phi_format);
  if (L->phi_format == LRQAT_PHI_FIXED_Q8) {
    if (L->bits < 2 || L->bits > 7) return fail(LRQAT_EINVAL, "fixed-point Phi0 needs 2 <= bits <= 7 (got %d)", L->bits);
  } else {
    if (L->bits < 2 || L->bits > 4) return fail(LRQAT_EINVAL, "packed INT-b Phi0 needs 2 <= bits <= 4 (got %d)", L->bits);
    if (L->in_features % 2) return fail(LRQAT_EINVAL, "packed INT-b Phi0 needs an even in_features");
  }
  if (L->group_size < 0) return fail(LRQAT_EINVAL, "group_size must be >= 0");
  if (L->group_size > 0) {
    if (L->in_features % L->group_size)
      return fail(LRQAT_EINVAL, "in_features %% group_size != 0 (%lld, %lld)", (long long)L->in_features,
                  (long long)L->group_size);
    // a 32-column chunk (the GEMM epilogue's unit of scale, mask and ds work) never straddles two groups
    if (L->group_size % 32)
      return fail(LRQAT_EUNSUPPORTED, "group_size must be a multiple of 32 (got %lld)", (long long)L->group_size);
  }
  if (L->act_dtype != LRQAT_FP32 && L->act_dtype != LRQAT_BF16) return fail(LRQAT_EINVAL, "unknown act_dtype");
  if (L->act_bits != 0 && L->act_bits != 8) return fail(LRQAT_EINVAL, "act_bits must be 0 or 8");
  if (L->act_bits == 8 && L->act_dtype != LRQAT_BF16)
    return fail(LRQAT_EUNSUPPORTED, "activation quantisation runs with bfloat16 activations only");
  d.m = L->out_features;
  d.k = L->in_features;
  d.r = L->rank;
  d.g = L->group_size;
  d.ngroups = d.g ? d.k / d.g : 1;
  d.kpad = round_up(d.k, GEMM_BN);
  d.mpad = round_up(d.m, GEMM_BM);
  d.bits = L->bits;
  d.packed = L->phi_format == LRQAT_PHI_INT_PACKED2;
  d.q8w = !d.packed && d.bits > 4;
  d.act = L->act_bits == 8;
  d.bf16 = L->act_dtype == LRQAT_BF16;
  d.c = L->alpha / float(L->rank);
  d.c64 = double(L->alpha) / double(L->rank);
  return LRQAT_OK;
}

enum Pass { kForward, kBackward, kInfer };

Workspace layout(const Dims& d, int64_t T, Pass pass) {
  Workspace w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += size_t(round_up(int64_t(bytes), 256));
    return at;
  };
  if (pass != kInfer) w.q = take(size_t(d.q8w ? d.m * d.kpad : d.m * d.kpad / 2));
  else if (d.k % 32) w.q = take(size_t(d.m * d.kpad / 2));  // merged weights re-laid with 16-byte aligned rows
  if (pass == kBackward) w.mask = take(size_t(d.m * (d.kpad / 16) * 2));
  if (d.act) {
    if (pass == kBackward) {
      w.xh = take(size_t(T * d.kpad * 2));  // X_hat in bfloat16 for the dW GEMM
    } else {
      w.n = take(size_t(T * d.kpad));
      w.sx = take(size_t(T * 4));
    }
  }
  if (pass == kBackward) {
    w.ds_part = take(size_t(d.m * (d.kpad / 32) * 4));
    if (d.bf16) {
      const int64_t ntn = (d.k + GEMM_BN - 1) / GEMM_BN, ntm = (d.m + GEMM_BM - 1) / GEMM_BM;
      w.dA_part = take(size_t(ntn * d.m * d.r * 4));
      w.dB_part = take(size_t(ntm * d.r * d.k * 4));
    } else {
      w.dW = take(size_t(d.m * d.k * 4));
    }
  }
  w.total = off;
  return w;
}

GridArgs grid_args(const Dims& d, const void* phi0, const float* A, const float* B, uint8_t* q, uint16_t* mask) {
  GridArgs a{};
  a.phi0 = static_cast<const uint8_t*>(phi0);
  a.ld_phi = d.packed ? d.k / 2 : d.k;
  a.A = A;
  a.B = B;
  a.m = d.m;
  a.k = d.k;
  a.r = int(d.r);
  a.c = d.c;
  a.c64 = d.c64;
  a.bits = d.bits;
  a.packed = d.packed;
  a.qout = q;
  a.q8out = d.q8w;
  a.ldq = d.q8w ? d.kpad : d.kpad / 2;
  a.kq = d.kpad;
  a.mout = mask;
  a.ldm = d.kpad / 16;
  return a;
}

lrqat_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return LRQAT_OK;
  return fail(LRQAT_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define LRQAT_TRY(expr)                         \
  do {                                          \
    const lrqat_status st_ = (expr);            \
    if (st_ != LRQAT_OK) return st_;            \
  } while (0)

#define NEED(ptr, align)                                                                        \
  do {                                                                                          \
    if (!(ptr)) return fail(LRQAT_EINVAL, "%s is NULL", #ptr);                                  \
    if (!aligned((ptr), (align))) return fail(LRQAT_EINVAL, "%s is not %d-byte aligned", #ptr, (align)); \
  } while (0)

// Y = X_hat (s (q - z))^T from the integer grid q [m][ldq] (int4 packed, or int8 when d.q8w).
lrqat_status weight_gemm_forward(const Dims& d, int64_t tokens, const void* X, const uint8_t* q, int64_t ldq,
                                 const float* s, const int32_t* z, void* Y, uint8_t* base, const Workspace& w,
                                 hipStream_t st) {
  if (!d.bf16) {
    F32Args fa{};
    fa.T = tokens; fa.m = d.m; fa.k = d.k; fa.r = int(d.r); fa.c = d.c;
    fa.X = static_cast<const float*>(X);
    fa.q = q; fa.ldq = ldq; fa.q8 = d.q8w;
    fa.s = s; fa.z = z; fa.gsize = d.g; fa.ngroups = d.ngroups;
    return hip_status(timed("f32_fwd", st, [&] { return launch_f32_forward(fa, static_cast<float*>(Y), st); }),
                      "f32_fwd");
  }
  int8_t* n = reinterpret_cast<int8_t*>(base + w.n);
  float* sx = reinterpret_cast<float*>(base + w.sx);
  if (d.act)
    LRQAT_TRY(hip_status(timed("act_quant", st, [&] {
                           return launch_act_quant(static_cast<const uint16_t*>(X), tokens, d.k, n, d.kpad, nullptr, 0,
                                                   sx, st);
                         }), "act_quant"));
  GemmArgs p{};
  p.M = tokens; p.N = d.m; p.K = d.k;
  p.a = d.act ? static_cast<const void*>(n) : X;
  p.lda = d.act ? d.kpad : d.k;
  p.b = q; p.ldb = ldq;
  p.s = s; p.z = z; p.gsize = d.g; p.ngroups = d.ngroups;
  p.sx = d.act ? sx : nullptr;
  p.out = Y; p.ldo = d.m;
  const int opt = (z ? kOptZ : 0) | (d.q8w ? kOptQ8 : 0);
  return hip_status(timed("gemm_fwd", st, [&] { return launch_gemm(kFwd, d.act, d.g != 0, opt, p, st); }), "gemm_fwd");
}

}  // namespace

extern "C" {

size_t lrqat_forward_workspace_size(const lrqat_layer* layer, int64_t tokens) {
  Dims d;
  if (check_layer(layer, d) != LRQAT_OK) return 0;
  if (tokens < 0 || tokens > kMaxDim) {
    fail(LRQAT_EINVAL, "tokens out of range");
    return 0;
  }
  return layout(d, tokens, kForward).total;
}

size_t lrqat_backward_workspace_size(const lrqat_layer* layer, int64_t tokens) {
  Dims d;
  if (check_layer(layer, d) != LRQAT_OK) return 0;
  if (tokens < 0 || tokens > kMaxDim) {
    fail(LRQAT_EINVAL, "tokens out of range");
    return 0;
  }
  return layout(d, tokens, kBackward).total;
}

lrqat_status lrqat_init_from_weights(const lrqat_layer* layer, const float* W0, float* s0_out, int32_t* z0_out,
                                     void* phi0_out, void* stream) {
  Dims d;
  LRQAT_TRY(check_layer(layer, d));
  NEED(W0, 4);
  NEED(s0_out, 4);
  if (z0_out && !aligned(z0_out, 4)) return fail(LRQAT_EINVAL, "z0_out is not 4-byte aligned");
  NEED(phi0_out, 16);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t gsize = d.g ? d.g : d.k;
  LRQAT_TRY(hip_status(timed("init_scale", st, [&] {
                         return launch_minmax_scale(W0, d.m, d.k, gsize, d.bits, s0_out, z0_out, st);
                       }), "init_scale"));
  LRQAT_TRY(hip_status(timed("init_encode", st, [&] {
                         return launch_encode(W0, s0_out, z0_out, d.m, d.k, gsize, d.bits, d.packed, phi0_out, st);
                       }), "init_encode"));
  return LRQAT_OK;
}

lrqat_status lrqat_forward(const lrqat_layer* layer, int64_t tokens, const void* X, const void* phi0, const float* s,
                           const int32_t* z, const float* A, const float* B, void* Y, void* ws, size_t ws_bytes,
                           void* stream) {
  Dims d;
  LRQAT_TRY(check_layer(layer, d));
  if (tokens < 0 || tokens > kMaxDim) return fail(LRQAT_EINVAL, "tokens out of range (%lld)", (long long)tokens);
  if (tokens == 0) return LRQAT_OK;
  NEED(X, 16);
  NEED(phi0, 16);
  NEED(s, 4);
  if (z && !aligned(z, 4)) return fail(LRQAT_EINVAL, "z is not 4-byte aligned");
  NEED(A, 4);
  NEED(B, 4);
  NEED(Y, 16);
  NEED(ws, 256);
  const Workspace w = layout(d, tokens, kForward);
  if (ws_bytes < w.total)
    return fail(LRQAT_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu bytes needed", ws_bytes, w.total);
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* base = static_cast<uint8_t*>(ws);
  uint8_t* q = base + w.q;
  const GridArgs ga = grid_args(d, phi0, A, B, q, nullptr);
  LRQAT_TRY(hip_status(timed("grid", st, [&] { return launch_grid(ga, st); }), "grid"));
  return weight_gemm_forward(d, tokens, X, q, ga.ldq, s, z, Y, base, w, st);
}

}  // extern "C"

namespace {

// The backward pass of lrqat_backward and lrqat_backward_static: `ws` is the
// caller's workspace or the library's device-resident scratch array.
lrqat_status backward_impl(const lrqat_layer* layer, int64_t tokens, const void* X, const void* phi0, const float* s,
                           const int32_t* z, const float* A, const float* B, const void* dY, void* dX, float* dA,
                           float* dB, float* ds, int accumulate, void* ws, size_t ws_bytes, void* stream) {
  Dims d;
  LRQAT_TRY(check_layer(layer, d));
  if (tokens < 0 || tokens > kMaxDim) return fail(LRQAT_EINVAL, "tokens out of range (%lld)", (long long)tokens);
  if (accumulate != 0 && accumulate != 1) return fail(LRQAT_EINVAL, "accumulate must be 0 or 1");
  NEED(dA, 4);
  NEED(dB, 4);
  if (ds && !aligned(ds, 4)) return fail(LRQAT_EINVAL, "ds is not 4-byte aligned");
  if (z && !aligned(z, 4)) return fail(LRQAT_EINVAL, "z is not 4-byte aligned");
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (tokens == 0) {
    LRQAT_TRY(hip_status(launch_reduce(nullptr, 0, d.m * d.r, dA, 0.f, accumulate, st), "reduce"));
    LRQAT_TRY(hip_status(launch_reduce(nullptr, 0, d.r * d.k, dB, 0.f, accumulate, st), "reduce"));
    if (ds) LRQAT_TRY(hip_status(launch_reduce(nullptr, 0, d.m * d.ngroups, ds, 0.f, accumulate, st), "reduce"));
    return LRQAT_OK;
  }
  NEED(X, 16);
  NEED(phi0, 16);
  NEED(s, 4);
  NEED(A, 4);
  NEED(B, 4);
  NEED(dY, 16);
  if (dX && !aligned(dX, 16)) return fail(LRQAT_EINVAL, "dX is not 16-byte aligned");
  NEED(ws, 256);
  const Workspace w = layout(d, tokens, kBackward);
  if (ws_bytes < w.total)
    return fail(LRQAT_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu bytes needed", ws_bytes, w.total);
  uint8_t* base = static_cast<uint8_t*>(ws);
  uint8_t* q = base + w.q;
  uint16_t* mask = reinterpret_cast<uint16_t*>(base + w.mask);
  const GridArgs ga = grid_args(d, phi0, A, B, q, mask);
  LRQAT_TRY(hip_status(timed("grid", st, [&] { return launch_grid(ga, st); }), "grid"));

  if (!d.bf16) {
    F32Args fa{};
    fa.T = tokens; fa.m = d.m; fa.k = d.k; fa.r = int(d.r); fa.c = d.c;
    fa.X = static_cast<const float*>(X);
    fa.dY = static_cast<const float*>(dY);
    fa.q = q; fa.ldq = ga.ldq; fa.q8 = d.q8w;
    fa.mask = mask; fa.ldm = ga.ldm;
    fa.s = s; fa.z = z; fa.gsize = d.g; fa.ngroups = d.ngroups;
    fa.A = A; fa.B = B;
    fa.dW = reinterpret_cast<float*>(base + w.dW);
    if (dX)
      LRQAT_TRY(hip_status(timed("f32_dx", st, [&] { return launch_f32_dx(fa, static_cast<float*>(dX), st); }), "f32_dx"));
    LRQAT_TRY(hip_status(timed("f32_dw", st, [&] { return launch_f32_dw(fa, dA, dB, ds, accumulate, st); }), "f32_dw"));
    return LRQAT_OK;
  }

  // W4A8: the dW GEMM runs on X_hat = s_x n, rounded to bfloat16
  uint16_t* xh = reinterpret_cast<uint16_t*>(base + w.xh);
  if (d.act)
    LRQAT_TRY(hip_status(timed("act_quant", st, [&] {
                           return launch_act_quant(static_cast<const uint16_t*>(X), tokens, d.k, nullptr, 0, xh,
                                                   d.kpad, nullptr, st);
                         }), "act_quant"));
  if (dX) {
    GemmArgs p{};
    p.M = tokens; p.N = d.k; p.K = d.m;
    p.a = dY; p.lda = d.m;
    p.b = q; p.ldb = ga.ldq;
    p.s = s; p.z = z; p.gsize = d.g; p.ngroups = d.ngroups;
    p.out = dX; p.ldo = d.k;
    const int opt = (z ? kOptZ : 0) | (d.q8w ? kOptQ8 : 0);
    LRQAT_TRY(hip_status(timed("gemm_dx", st, [&] { return launch_gemm(kDx, false, d.g != 0, opt, p, st); }),
                         "gemm_dx"));
  }
  float* dA_part = reinterpret_cast<float*>(base + w.dA_part);
  float* dB_part = reinterpret_cast<float*>(base + w.dB_part);
  float* ds_part = reinterpret_cast<float*>(base + w.ds_part);
  GemmArgs p{};
  p.M = d.m; p.N = d.k; p.K = tokens;
  p.a = dY; p.lda = d.m;
  p.b = d.act ? static_cast<const void*>(xh) : X;
  p.ldb = d.act ? d.kpad : d.k;
  p.s = s; p.z = z; p.gsize = d.g; p.ngroups = d.ngroups;
  p.mask = mask; p.ldm = ga.ldm;
  p.Am = A; p.Bm = B; p.r = int(d.r);
  p.dA_part = dA_part; p.dB_part = dB_part;
  if (ds) {
    p.qd = q; p.ldqd = ga.ldq; p.qd8 = d.q8w;
    p.ds_part = ds_part; p.ldds = d.kpad / 32;
  }
  LRQAT_TRY(hip_status(timed("gemm_dw", st, [&] { return launch_gemm(kDw, false, d.g != 0, 0, p, st); }), "gemm_dw"));
  const int64_t ntn = (d.k + GEMM_BN - 1) / GEMM_BN, ntm = (d.m + GEMM_BM - 1) / GEMM_BM;
  Reduce2Args ra{};
  ra.part[0] = dA_part; ra.nparts[0] = ntn; ra.n[0] = d.m * d.r; ra.out[0] = dA;
  ra.part[1] = dB_part; ra.nparts[1] = ntm; ra.n[1] = d.r * d.k; ra.out[1] = dB;
  for (int i = 0; i < 2; ++i) ra.vec[i] = ra.n[i] % 4 == 0 && aligned(ra.out[i], 16);
  ra.c = d.c;
  ra.accumulate = accumulate;
  LRQAT_TRY(hip_status(timed("reduce", st, [&] { return launch_reduce2(ra, st); }), "reduce"));
  if (ds) {
    const int64_t nchunks = (d.k + 31) / 32, cpg = d.g ? d.g / 32 : nchunks;
    LRQAT_TRY(hip_status(timed("reduce_ds", st, [&] {
                           return launch_reduce_ds(ds_part, d.m, d.kpad / 32, nchunks, cpg, d.ngroups, ds, accumulate, st);
                         }), "reduce_ds"));
  }
  return LRQAT_OK;
}

// ---- the device-resident scratch of lrqat_backward_static
// One array per GPU (each device holds its own copy of a __device__ variable),
// kept until the process ends.  Host code never passes `scratch` itself to a
// kernel: its device address is looked up once per device.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

namespace {

lrqat_status static_scratch(void** out) {
  int dev = 0;
  LRQAT_TRY(hip_status(hipGetDevice(&dev), "hipGetDevice"));
  if (dev < 0 || dev >= kMaxDevices) return fail(LRQAT_EINVAL, "device %d beyond the %d this library tracks", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    LRQAT_TRY(hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)"));
    if (!p) return fail(LRQAT_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LRQAT_OK;
}

}  // namespace

extern "C" {

lrqat_status lrqat_backward(const lrqat_layer* layer, int64_t tokens, const void* X, const void* phi0, const float* s,
                            const int32_t* z, const float* A, const float* B, const void* dY, void* dX, float* dA,
                            float* dB, float* ds, int accumulate, void* ws, size_t ws_bytes, void* stream) {
  return backward_impl(layer, tokens, X, phi0, s, z, A, B, dY, dX, dA, dB, ds, accumulate, ws, ws_bytes, stream);
}

lrqat_status lrqat_backward_static(const lrqat_layer* layer, int64_t tokens, const void* X, const void* phi0,
                                   const float* s, const int32_t* z, const float* A, const float* B, const void* dY,
                                   void* dX, float* dA, float* dB, float* ds, int accumulate, void* stream) {
  Dims d;
  LRQAT_TRY(check_layer(layer, d));
  if (tokens < 0 || tokens > kMaxDim) return fail(LRQAT_EINVAL, "tokens out of range (%lld)", (long long)tokens);
  const size_t need = layout(d, tokens, kBackward).total;
  if (need > kStaticScratchBytes)
    return fail(LRQAT_EWORKSPACE,
                "lrqat_backward_static: this layer needs %zu bytes of scratch, more than the %zu bytes of the "
                "library's device array; use lrqat_backward with a workspace",
                need, kStaticScratchBytes);
  void* ws = nullptr;
  LRQAT_TRY(static_scratch(&ws));
  return backward_impl(layer, tokens, X, phi0, s, z, A, B, dY, dX, dA, dB, ds, accumulate, ws, kStaticScratchBytes,
                       stream);
}

size_t lrqat_backward_static_capacity(void) { return kStaticScratchBytes; }

lrqat_status lrqat_merge_to_int4(const lrqat_layer* layer, const void* phi0, const float* A, const float* B,
                                 uint8_t* W_int4, void* stream) {
  Dims d;
  LRQAT_TRY(check_layer(layer, d));
  if (d.k % 2) return fail(LRQAT_EINVAL, "merge_to_int4 needs an even in_features");
  if (d.bits > 4) return fail(LRQAT_EINVAL, "merge_to_int4 needs bits <= 4 (got %d)", d.bits);
  NEED(phi0, 16);
  NEED(A, 4);
  NEED(B, 4);
  NEED(W_int4, 16);
  hipStream_t st = static_cast<hipStream_t>(stream);
  GridArgs ga = grid_args(d, phi0, A, B, W_int4, nullptr);
  ga.ldq = d.k / 2;
  ga.kq = d.k;
  LRQAT_TRY(hip_status(timed("merge", st, [&] { return launch_grid(ga, st); }), "merge"));
  return LRQAT_OK;
}

lrqat_status lrqat_init_lp(const lrqat_layer* layer, const float* W0, float p, int n_grid, float* s0_out,
                           void* phi0_out, void* stream) {
  Dims d;
  LRQAT_TRY(check_layer(layer, d));
  NEED(W0, 4);
  NEED(s0_out, 4);
  NEED(phi0_out, 16);
  if (!(p >= 1.f && p <= 16.f)) return fail(LRQAT_EINVAL, "p must be in [1, 16] (got %g)", double(p));
  if (n_grid < 1 || n_grid > 10000) return fail(LRQAT_EINVAL, "n_grid must be in [1, 10000] (got %d)", n_grid);
  const int64_t gsize = d.g ? d.g : d.k;
  if (gsize > kLpMaxGroup)
    return fail(LRQAT_EUNSUPPORTED, "the L^p search holds a row or group of at most %lld weights (got %lld)",
                (long long)kLpMaxGroup, (long long)gsize);
  hipStream_t st = static_cast<hipStream_t>(stream);
  LRQAT_TRY(hip_status(timed("init_lp", st, [&] {
                         return launch_lp_search(W0, d.m, d.k, gsize, d.bits, p, n_grid, s0_out, nullptr, st);
                       }), "init_lp"));
  LRQAT_TRY(hip_status(timed("init_encode", st, [&] {
                         return launch_encode(W0, s0_out, nullptr, d.m, d.k, gsize, d.bits, d.packed, phi0_out, st);
                       }), "init_encode"));
  return LRQAT_OK;
}

static lrqat_status loftq_dims(const lrqat_layer* layer, Dims& d, int& l) {
  LRQAT_TRY(check_layer(layer, d));
  if (!d.packed) return fail(LRQAT_EINVAL, "LoftQ initialisation writes INT-b Phi0: phi_format must be INT_PACKED2");
  if (d.r > kLoftqMaxRank)
    return fail(LRQAT_EUNSUPPORTED, "LoftQ initialisation runs ranks up to %d (got %lld)", kLoftqMaxRank,
                (long long)d.r);
  l = int(std::min<int64_t>(d.r + kLoftqOversample, std::min(d.m, d.k)));
  if (l < d.r) return fail(LRQAT_EINVAL, "rank %lld exceeds min(m, k)", (long long)d.r);
  if (d.alpha_nonpos()) return fail(LRQAT_EINVAL, "LoftQ initialisation needs alpha / r > 0");
  return LRQAT_OK;
}

size_t lrqat_init_loftq_workspace_size(const lrqat_layer* layer) {
  Dims d;
  int l = 0;
  if (loftq_dims(layer, d, l) != LRQAT_OK) return 0;
  return loftq_workspace(d.m, d.k, l);
}

lrqat_status lrqat_init_loftq(const lrqat_layer* layer, const float* W0, const float* s0, int n_iter, void* phi0_out,
                              float* A_out, float* B_out, float* sigma_out, void* ws, size_t ws_bytes, void* stream) {
  Dims d;
  int l = 0;
  LRQAT_TRY(loftq_dims(layer, d, l));
  NEED(W0, 4);
  NEED(s0, 4);
  NEED(phi0_out, 16);
  NEED(A_out, 4);
  NEED(B_out, 4);
  if (sigma_out && !aligned(sigma_out, 4)) return fail(LRQAT_EINVAL, "sigma_out is not 4-byte aligned");
  if (n_iter < 0 || n_iter > 1000) return fail(LRQAT_EINVAL, "n_iter must be in [0, 1000] (got %d)", n_iter);
  NEED(ws, 256);
  const size_t need = loftq_workspace(d.m, d.k, l);
  if (ws_bytes < need)
    return fail(LRQAT_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu bytes needed", ws_bytes, need);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t gsize = d.g ? d.g : d.k;
  return hip_status(timed("init_loftq", st, [&] {
                      return launch_loftq(W0, s0, d.m, d.k, gsize, d.bits, int(d.r), l, d.c64, n_iter,
                                          static_cast<uint8_t*>(phi0_out), A_out, B_out, sigma_out, ws, st);
                    }), "init_loftq");
}

size_t lrqat_infer_workspace_size(const lrqat_layer* layer, int64_t tokens) {
  Dims d;
  if (check_layer(layer, d) != LRQAT_OK) return 0;
  if (tokens < 0 || tokens > kMaxDim) {
    fail(LRQAT_EINVAL, "tokens out of range");
    return 0;
  }
  return std::max<size_t>(layout(d, tokens, kInfer).total, 256);
}

lrqat_status lrqat_infer_forward(const lrqat_layer* layer, int64_t tokens, const void* X, const uint8_t* W_int4,
                                 const float* s, const int32_t* z, void* Y, void* ws, size_t ws_bytes, void* stream) {
  Dims d;
  LRQAT_TRY(check_layer(layer, d));
  if (d.k % 2) return fail(LRQAT_EINVAL, "merged int4 weights need an even in_features");
  if (d.bits > 4) return fail(LRQAT_EINVAL, "merged int4 weights need bits <= 4 (got %d)", d.bits);
  if (tokens < 0 || tokens > kMaxDim) return fail(LRQAT_EINVAL, "tokens out of range (%lld)", (long long)tokens);
  if (tokens == 0) return LRQAT_OK;
  NEED(X, 16);
  NEED(W_int4, 16);
  NEED(s, 4);
  if (z && !aligned(z, 4)) return fail(LRQAT_EINVAL, "z is not 4-byte aligned");
  NEED(Y, 16);
  NEED(ws, 256);
  const Workspace w = layout(d, tokens, kInfer);
  if (ws_bytes < w.total)
    return fail(LRQAT_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu bytes needed", ws_bytes, w.total);
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* base = static_cast<uint8_t*>(ws);
  Dims di = d;
  di.q8w = 0;  // merged weights are always packed int4
  const uint8_t* q = W_int4;
  int64_t ldq = d.k / 2;
  if (d.k % 32) {
    // rows of k/2 bytes are not 16-byte aligned: copy them into zero-padded rows of kpad/2 bytes
    uint8_t* qp = base + w.q;
    LRQAT_TRY(hip_status(timed("infer_relayout", st, [&] {
                           return launch_repack_rows(W_int4, d.m, d.k / 2, qp, d.kpad / 2, st);
                         }), "infer_relayout"));
    q = qp;
    ldq = d.kpad / 2;
  }
  return weight_gemm_forward(di, tokens, X, q, ldq, s, z, Y, base, w, st);
}

static lrqat_status adamw_args(const lrqat_adamw_config* cfg, int n_groups, const lrqat_param_group* groups,
                               OptimArgs& a) {
  if (!cfg) return fail(LRQAT_EINVAL, "config is NULL");
  if (n_groups < 0 || n_groups > kMaxOptimGroups)
    return fail(LRQAT_EINVAL, "n_groups must be in [0, %d] (got %d)", kMaxOptimGroups, n_groups);
  if (n_groups && !groups) return fail(LRQAT_EINVAL, "groups is NULL");
  if (!(cfg->beta1 >= 0.f && cfg->beta1 < 1.f && cfg->beta2 >= 0.f && cfg->beta2 < 1.f))
    return fail(LRQAT_EINVAL, "betas must be in [0, 1)");
  if (!(cfg->eps >= 0.f) || !std::isfinite(cfg->eps) || !std::isfinite(cfg->max_grad_norm))
    return fail(LRQAT_EINVAL, "eps and max_grad_norm must be finite, eps >= 0");
  if (cfg->total_steps < 1 || cfg->warmup_steps < 0 || cfg->warmup_steps > cfg->total_steps)
    return fail(LRQAT_EINVAL, "need 0 <= warmup_steps <= total_steps and total_steps >= 1");
  a = OptimArgs{};
  a.ngroups = n_groups;
  a.total = cfg->total_steps;
  a.warmup = cfg->warmup_steps;
  a.beta1 = cfg->beta1;
  a.beta2 = cfg->beta2;
  a.eps = cfg->eps;
  a.max_norm = cfg->max_grad_norm;
  for (int i = 0; i < n_groups; ++i) {
    const lrqat_param_group& g = groups[i];
    if (g.n < 0) return fail(LRQAT_EINVAL, "group %d: n < 0", i);
    if (g.n > 0 && (!g.param || !g.grad || !g.exp_avg || !g.exp_avg_sq))
      return fail(LRQAT_EINVAL, "group %d: a NULL tensor", i);
    if (!aligned(g.param, 4) || !aligned(g.grad, 4) || !aligned(g.exp_avg, 4) || !aligned(g.exp_avg_sq, 4))
      return fail(LRQAT_EINVAL, "group %d: tensors must be 4-byte aligned", i);
    if (!std::isfinite(g.lr_max) || !std::isfinite(g.weight_decay))
      return fail(LRQAT_EINVAL, "group %d: lr_max and weight_decay must be finite", i);
    a.g[i] = OptimGroup{g.param, g.grad, g.exp_avg, g.exp_avg_sq, g.n, g.lr_max, g.weight_decay};
  }
  optim_prepare(a);
  return LRQAT_OK;
}

size_t lrqat_adamw_workspace_size(int n_groups, const lrqat_param_group* groups) {
  lrqat_adamw_config cfg{0.9f, 0.95f, 1e-8f, 1.f, 1, 0};
  OptimArgs a;
  if (adamw_args(&cfg, n_groups, groups, a) != LRQAT_OK) return 0;
  return size_t(round_up(int64_t(optim_chunks(a) * 8 + 16), 256));
}

lrqat_status lrqat_adamw_step(const lrqat_adamw_config* cfg, int64_t step, int n_groups,
                              const lrqat_param_group* groups, float* grad_norm_out, void* ws, size_t ws_bytes,
                              void* stream) {
  OptimArgs a;
  LRQAT_TRY(adamw_args(cfg, n_groups, groups, a));
  if (step < 1) return fail(LRQAT_EINVAL, "step is 1-based (got %lld)", (long long)step);
  a.step = step;
  if (grad_norm_out && !aligned(grad_norm_out, 4)) return fail(LRQAT_EINVAL, "grad_norm_out is not 4-byte aligned");
  NEED(ws, 256);
  const size_t need = size_t(round_up(int64_t(optim_chunks(a) * 8 + 16), 256));
  if (ws_bytes < need) return fail(LRQAT_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu bytes needed",
                                   ws_bytes, need);
  double* part = reinterpret_cast<double*>(static_cast<uint8_t*>(ws) + 16);
  float* norm_coef = static_cast<float*>(ws);
  hipStream_t st = static_cast<hipStream_t>(stream);
  return hip_status(timed("adamw", st, [&] { return launch_adamw(a, part, norm_coef, grad_norm_out, st); }), "adamw");
}

const char* lrqat_status_string(lrqat_status status) {
  switch (status) {
    case LRQAT_OK: return "LRQAT_OK";
    case LRQAT_EINVAL: return "LRQAT_EINVAL";
    case LRQAT_EUNSUPPORTED: return "LRQAT_EUNSUPPORTED";
    case LRQAT_EWORKSPACE: return "LRQAT_EWORKSPACE";
    case LRQAT_EHIP: return "LRQAT_EHIP";
  }
  return "LRQAT_UNKNOWN";
}

const char* lrqat_last_error(void) { return g_last_error.c_str(); }

void lrqat_timing_enable(int enable) {
  std::lock_guard<std::mutex> lk(g_timing_mu);
  g_timing = enable != 0;
}

void lrqat_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_timing_mu);
  for (auto& p : g_pending) {
    (void)hipEventSynchronize(p.stop);
    (void)hipEventDestroy(p.start);
    (void)hipEventDestroy(p.stop);
  }
  g_pending.clear();
  g_totals.clear();
}

int lrqat_timing_read(const char** names, int64_t* launches, double* total_ms, int max_kernels) {
  std::lock_guard<std::mutex> lk(g_timing_mu);
  int rc = 0;
  for (auto& p : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.stop) != hipSuccess || hipEventElapsedTime(&ms, p.start, p.stop) != hipSuccess) rc = -1;
    auto& slot = g_totals[p.name];
    slot.first = p.name;
    slot.second.launches += 1;
    slot.second.ms += ms;
    (void)hipEventDestroy(p.start);
    (void)hipEventDestroy(p.stop);
  }
  g_pending.clear();
  if (rc) return rc;
  int i = 0;
  for (auto& kv : g_totals) {
    if (i >= max_kernels) break;
    if (names) names[i] = kv.second.first;
    if (launches) launches[i] = kv.second.second.launches;
    if (total_ms) total_ms[i] = kv.second.second.ms;
    ++i;
  }
  return i;
}

}  // extern "C"
