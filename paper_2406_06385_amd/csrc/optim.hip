// The optimizer step after the backward pass (Appendix B, Table B1): AdamW
// (decoupled weight decay) over the trainable tensors A, B and s, with global
// L2-norm gradient clipping and a linear warm-up / linear decay learning-rate
// schedule.  Three launches, all bandwidth-bound:
//   1. k_sq_partials: fixed-size chunks of every group's gradient, sum of
//      squares in float64 per chunk (deterministic partition and order);
//   2. k_norm_finalize: one block adds the chunk sums in order and writes the
//      norm and the clip coefficient min(1, max_norm / (norm + 1e-6));
//   3. k_adamw: the elementwise update, 16-byte vectors where aligned.
#include "kernels.h"

namespace lrqat {

constexpr int OPT_THREADS = 256;
constexpr int64_t OPT_CHUNK = 8192;  // gradient elements per partial sum

__device__ __forceinline__ int group_of(const OptimArgs& a, int64_t idx, int64_t* first) {
  int g = 0;
  while (g + 1 < a.ngroups && idx >= a.first[g + 1]) ++g;
  *first = a.first[g];
  return g;
}

// One block per chunk: sum of g^2 over elements [c * CHUNK, (c + 1) * CHUNK) of its group.
__global__ __launch_bounds__(OPT_THREADS) void k_sq_partials(OptimArgs a, double* __restrict__ part) {
  int64_t first;
  const int g = group_of(a, blockIdx.x, &first);
  const OptimGroup& G = a.g[g];
  const int64_t c = blockIdx.x - first;
  const int64_t lo = c * OPT_CHUNK, hi = min(G.n, lo + OPT_CHUNK);
  double acc = 0.0;
  if ((reinterpret_cast<uintptr_t>(G.grad) & 15) == 0) {
    // 16-byte vectors (chunks start at multiples of 8192 elements), then the tail
    const int64_t nv = (hi - lo) / 4;
    double acc1 = 0.0;
    for (int64_t i = threadIdx.x; i < nv; i += OPT_THREADS) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(G.grad + lo + 4 * i);
      acc = __builtin_fma(double(v[0]), double(v[0]), acc);
      acc1 = __builtin_fma(double(v[1]), double(v[1]), acc1);
      acc = __builtin_fma(double(v[2]), double(v[2]), acc);
      acc1 = __builtin_fma(double(v[3]), double(v[3]), acc1);
    }
    acc += acc1;
    for (int64_t j = lo + 4 * nv + threadIdx.x; j < hi; j += OPT_THREADS) {
      const double x = G.grad[j];
      acc = __builtin_fma(x, x, acc);
    }
  } else {
    for (int64_t j = lo + threadIdx.x; j < hi; j += OPT_THREADS) {
      const double x = G.grad[j];
      acc = __builtin_fma(x, x, acc);
    }
  }
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  __shared__ double red[OPT_THREADS / 64];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

// norm_coef[0] = ||g||_2, norm_coef[1] = clip coefficient (1 without clipping).
__global__ __launch_bounds__(OPT_THREADS) void k_norm_finalize(const double* __restrict__ part, int64_t nparts,
                                                               float max_norm, float* __restrict__ norm_coef,
                                                               float* __restrict__ norm_out) {
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < nparts; i += OPT_THREADS) acc += part[i];
  __shared__ double red[OPT_THREADS];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = OPT_THREADS / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double norm = __builtin_sqrt(red[0]);
    const double coef = max_norm > 0.f ? fmin(1.0, double(max_norm) / (norm + 1e-6)) : 1.0;
    norm_coef[0] = float(norm);
    norm_coef[1] = float(coef);
    if (norm_out) *norm_out = float(norm);
  }
}

// b^t for an integer step t >= 0 by binary exponentiation (float64).
__device__ __forceinline__ double ipow(double b, int64_t t) {
  double r = 1.0;
  while (t > 0) {
    if (t & 1) r *= b;
    b *= b;
    t >>= 1;
  }
  return r;
}

// One element of the update; lr, the bias corrections and the clip coefficient are per call.
struct AdamStep {
  float lr, wd, b1, b2, eps, inv_bc1, inv_sqrt_bc2, coef;
  __device__ __forceinline__ void operator()(float& p, float g, float& m, float& v) const {
    g *= coef;
    p *= 1.f - lr * wd;
    m = b1 * m + (1.f - b1) * g;
    v = b2 * v + (1.f - b2) * g * g;
    const float denom = __builtin_sqrtf(v) * inv_sqrt_bc2 + eps;
    p -= lr * (m * inv_bc1) / denom;
  }
};

// Grid-stride elementwise update over all groups; a block works inside one group.
__global__ __launch_bounds__(OPT_THREADS) void k_adamw(OptimArgs a, const float* __restrict__ norm_coef) {
  int64_t first;
  const int g = group_of(a, blockIdx.x, &first);
  const OptimGroup& G = a.g[g];
  // schedule (linear warm-up over the first W steps, then linear decay to zero at N), t = step - 1
  const double t = double(a.step - 1);
  double f;
  if (t < double(a.warmup)) f = t / double(a.warmup > 0 ? a.warmup : 1);
  else f = fmax(0.0, (double(a.total) - t) / double(a.total - a.warmup > 0 ? a.total - a.warmup : 1));
  AdamStep st;
  st.lr = float(double(G.lr_max) * f);
  st.wd = G.weight_decay;
  st.b1 = a.beta1;
  st.b2 = a.beta2;
  st.eps = a.eps;
  st.inv_bc1 = float(1.0 / (1.0 - ipow(double(a.beta1), a.step)));
  st.inv_sqrt_bc2 = float(1.0 / __builtin_sqrt(1.0 - ipow(double(a.beta2), a.step)));
  st.coef = norm_coef[1];
  const int64_t c = blockIdx.x - first;
  const int64_t lo = c * OPT_CHUNK, hi = min(G.n, lo + OPT_CHUNK);
  const bool vec = ((reinterpret_cast<uintptr_t>(G.param) | reinterpret_cast<uintptr_t>(G.grad) |
                     reinterpret_cast<uintptr_t>(G.exp_avg) | reinterpret_cast<uintptr_t>(G.exp_avg_sq)) & 15) == 0;
  if (vec) {
    const int64_t nv = (hi - lo) / 4;
    for (int64_t i = threadIdx.x; i < nv; i += OPT_THREADS) {
      const int64_t j = lo + 4 * i;
      f32x4 p = *reinterpret_cast<const f32x4*>(G.param + j);
      const f32x4 gg = *reinterpret_cast<const f32x4*>(G.grad + j);
      f32x4 m = *reinterpret_cast<const f32x4*>(G.exp_avg + j);
      f32x4 v = *reinterpret_cast<const f32x4*>(G.exp_avg_sq + j);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float pe = p[e], me = m[e], ve = v[e];
        st(pe, gg[e], me, ve);
        p[e] = pe;
        m[e] = me;
        v[e] = ve;
      }
      *reinterpret_cast<f32x4*>(G.param + j) = p;
      *reinterpret_cast<f32x4*>(G.exp_avg + j) = m;
      *reinterpret_cast<f32x4*>(G.exp_avg_sq + j) = v;
    }
    for (int64_t j = lo + 4 * nv + threadIdx.x; j < hi; j += OPT_THREADS) st(G.param[j], G.grad[j], G.exp_avg[j], G.exp_avg_sq[j]);
  } else {
    for (int64_t j = lo + threadIdx.x; j < hi; j += OPT_THREADS) st(G.param[j], G.grad[j], G.exp_avg[j], G.exp_avg_sq[j]);
  }
}

int64_t optim_chunks(const OptimArgs& a) { return a.ngroups ? a.first[a.ngroups] : 0; }

void optim_prepare(OptimArgs& a) {
  int64_t total = 0;
  for (int g = 0; g < a.ngroups; ++g) {
    a.first[g] = total;
    total += (a.g[g].n + OPT_CHUNK - 1) / OPT_CHUNK;
  }
  a.first[a.ngroups] = total;
}

hipError_t launch_adamw(const OptimArgs& a, double* part, float* norm_coef, float* norm_out, hipStream_t st) {
  const int64_t nc = optim_chunks(a);
  if (nc > 0) {
    k_sq_partials<<<unsigned(nc), OPT_THREADS, 0, st>>>(a, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  k_norm_finalize<<<1, OPT_THREADS, 0, st>>>(part, nc, a.max_norm, norm_coef, norm_out);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nc == 0) return e;
  k_adamw<<<unsigned(nc), OPT_THREADS, 0, st>>>(a, norm_coef);
  return hipGetLastError();
}

}  // namespace lrqat
