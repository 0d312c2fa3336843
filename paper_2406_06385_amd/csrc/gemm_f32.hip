// float32-activation path of the LR-QAT layer ("FP32 compute data type",
// Section 4.2).  The same integer grid and clip mask as the bfloat16 path feed
// plain float32 FMA tiles; dW = dY^T X is kept in the workspace, and
// G = s * M * dW is formed on the fly by the tile kernel that contracts it
// with B^T and A^T.  A correctness path: the workloads run in bfloat16.
#include "kernels.h"

namespace lrqat {

constexpr int F_T = 64, F_K = 16;

// C[M][N] = sum_K a(i, kk) b(kk, j); block tile 64 x 64, 256 threads with 4 x 4 outputs each.
template <class OA, class OB, class EP>
__global__ __launch_bounds__(256) void k_f32_gemm(int64_t M, int64_t N, int64_t K, OA oa, OB ob, EP ep) {
  __shared__ float As[F_K][F_T + 4], Bs[F_K][F_T + 4];
  const int64_t ntn = (N + F_T - 1) / F_T;
  const int64_t m0 = int64_t(blockIdx.x / ntn) * F_T, n0 = int64_t(blockIdx.x % ntn) * F_T;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float c[4][4] = {};
  for (int64_t k0 = 0; k0 < K; k0 += F_K) {
    for (int q = 0; q < 4; ++q) {
      const int e = threadIdx.x + 256 * q;
      const int kk = e >> 6, x = e & 63;
      As[kk][x] = (m0 + x < M && k0 + kk < K) ? oa(m0 + x, k0 + kk) : 0.f;
      Bs[kk][x] = (n0 + x < N && k0 + kk < K) ? ob(k0 + kk, n0 + x) : 0.f;
    }
    __syncthreads();
    for (int kk = 0; kk < F_K; ++kk) {
      float a[4], b[4];
      for (int d = 0; d < 4; ++d) {
        a[d] = As[kk][4 * ty + d];
        b[d] = Bs[kk][4 * tx + d];
      }
      for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) c[i][j] = __builtin_fmaf(a[i], b[j], c[i][j]);
    }
    __syncthreads();
  }
  for (int i = 0; i < 4; ++i)
    for (int j = 0; j < 4; ++j) {
      const int64_t row = m0 + 4 * ty + i, col = n0 + 4 * tx + j;
      if (row < M && col < N) ep(row, col, c[i][j]);
    }
}

struct WeightHat {  // s(i, j) * (q(i, j) - z(i, j)) from the integer grid
  const uint8_t* q;
  int64_t ldq;
  int q8;
  const float* s;
  const int32_t* z;
  int64_t gsize, ngroups;
  __device__ int grid(int64_t i, int64_t j) const {
    if (q8) return int(int8_t(q[i * ldq + j]));
    const uint32_t byte = q[i * ldq + (j >> 1)];
    return int(byte << (28 - 4 * int(j & 1))) >> 28;
  }
  __device__ float operator()(int64_t i, int64_t j) const {
    const int64_t gi = gsize ? i * ngroups + j / gsize : i;
    const int zz = z ? z[gi] : 0;
    return float(grid(i, j) - zz) * s[gi];
  }
};

struct Mat {  // a(i, j) = p[i * ld + j]
  const float* p;
  int64_t ld;
  __device__ float operator()(int64_t i, int64_t j) const { return p[i * ld + j]; }
};
struct MatT {  // a(i, j) = p[j * ld + i]
  const float* p;
  int64_t ld;
  __device__ float operator()(int64_t i, int64_t j) const { return p[j * ld + i]; }
};
struct WeightHatT {
  WeightHat w;
  __device__ float operator()(int64_t kk, int64_t i) const { return w(i, kk); }
};

struct StoreOut {
  float* p;
  int64_t ld;
  __device__ void operator()(int64_t i, int64_t j, float v) const { p[i * ld + j] = v; }
};
struct GHat {  // G(i, j) = s M dW from the stored dW
  const float* dw;
  int64_t k;
  const uint16_t* mask;
  int64_t ldm;
  const float* s;
  int64_t gsize, ngroups;
  __device__ float operator()(int64_t i, int64_t j) const {
    const int bit = (mask[i * ldm + (j >> 4)] >> (j & 15)) & 1;
    const float sc = gsize ? s[i * ngroups + j / gsize] : s[i];
    return bit ? dw[i * k + j] * sc : 0.f;
  }
};
struct StoreGrad {  // out = (accumulate ? out : 0) + c * v
  float* p;
  int64_t ld;
  float c;
  int accumulate;
  __device__ void operator()(int64_t i, int64_t j, float v) const {
    float* d = p + i * ld + j;
    *d = (accumulate ? *d : 0.f) + c * v;
  }
};

template <class OA, class OB, class EP>
static hipError_t run(int64_t M, int64_t N, int64_t K, OA oa, OB ob, EP ep, hipStream_t st) {
  const int64_t nblocks = ((N + F_T - 1) / F_T) * ((M + F_T - 1) / F_T);
  if (nblocks == 0) return hipSuccess;
  k_f32_gemm<<<unsigned(nblocks), 256, 0, st>>>(M, N, K, oa, ob, ep);
  return hipGetLastError();
}

static WeightHat weight(const F32Args& a) { return WeightHat{a.q, a.ldq, a.q8, a.s, a.z, a.gsize, a.ngroups}; }

hipError_t launch_f32_forward(const F32Args& a, float* Y, hipStream_t st) {
  // Y[t][i] = sum_j X[t][j] W_hat[i][j]
  return run(a.T, a.m, a.k, Mat{a.X, a.k}, WeightHatT{weight(a)}, StoreOut{Y, a.m}, st);
}

hipError_t launch_f32_dx(const F32Args& a, float* dX, hipStream_t st) {
  // dX[t][j] = sum_i dY[t][i] W_hat[i][j]
  return run(a.T, a.k, a.m, Mat{a.dY, a.m}, weight(a), StoreOut{dX, a.k}, st);
}

// ds[i][grp] = (accumulate ? ds : 0) + sum over the group's columns of dW (q - z); one thread per (row, group).
__global__ __launch_bounds__(256) void k_f32_ds(WeightHat w, const float* __restrict__ dw, int64_t m, int64_t k,
                                                float* __restrict__ ds, int accumulate) {
  const int64_t ng = w.gsize ? w.ngroups : 1;
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= m * ng) return;
  const int64_t i = idx / ng, grp = idx % ng;
  const int64_t j0 = w.gsize ? grp * w.gsize : 0, j1 = w.gsize ? j0 + w.gsize : k;
  const int zz = w.z ? w.z[idx] : 0;
  float acc = 0.f;
  for (int64_t j = j0; j < j1; ++j) acc = __builtin_fmaf(dw[i * k + j], float(w.grid(i, j) - zz), acc);
  ds[idx] = (accumulate ? ds[idx] : 0.f) + acc;
}

hipError_t launch_f32_dw(const F32Args& a, float* dA, float* dB, float* ds, int accumulate, hipStream_t st) {
  // dW[i][j] = sum_t dY[t][i] X[t][j]
  hipError_t e = run(a.m, a.k, a.T, MatT{a.dY, a.m}, Mat{a.X, a.k}, StoreOut{a.dW, a.k}, st);
  if (e != hipSuccess) return e;
  const GHat g{a.dW, a.k, a.mask, a.ldm, a.s, a.gsize, a.ngroups};
  // dA[i][rho] = c sum_j G[i][j] B[rho][j]
  e = run(a.m, int64_t(a.r), a.k, g, MatT{a.B, a.k}, StoreGrad{dA, a.r, a.c, accumulate}, st);
  if (e != hipSuccess) return e;
  // dB[rho][j] = c sum_i A[i][rho] G[i][j]
  e = run(int64_t(a.r), a.k, a.m, MatT{a.A, a.r}, g, StoreGrad{dB, a.k, a.c, accumulate}, st);
  if (e != hipSuccess || !ds) return e;
  const int64_t n = a.m * (a.gsize ? a.ngroups : 1);
  k_f32_ds<<<unsigned((n + 255) / 256), 256, 0, st>>>(weight(a), a.dW, a.m, a.k, ds, accumulate);
  return hipGetLastError();
}

}  // namespace lrqat
