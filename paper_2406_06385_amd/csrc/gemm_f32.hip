// float32-activation path of the LR-QAT layer ("FP32 compute data type",
// Section 4.2).  The same packed integer grid and clip mask as the bfloat16
// path feed plain float32 FMA tiles; G = s * M * dY^T X is staged in the
// workspace and contracted with B^T and A^T by the same tile kernel.
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

struct WeightHat {  // s(i, j) * q(i, j) from the packed grid
  const uint8_t* q;
  int64_t ldq;
  const float* s;
  int64_t gsize, ngroups;
  __device__ float operator()(int64_t i, int64_t j) const {
    const uint32_t byte = q[i * ldq + (j >> 1)];
    const int v = int(byte << (28 - 4 * int(j & 1))) >> 28;
    const float sc = gsize ? s[i * ngroups + j / gsize] : s[i];
    return float(v) * sc;
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
struct StoreG {  // G = s * M * dW
  float* g;
  int64_t k;
  const uint16_t* mask;
  int64_t ldm;
  const float* s;
  int64_t gsize, ngroups;
  __device__ void operator()(int64_t i, int64_t j, float v) const {
    const int bit = (mask[(i >> 4) * ldm + j] >> (i & 15)) & 1;
    const float sc = gsize ? s[i * ngroups + j / gsize] : s[i];
    g[i * k + j] = bit ? v * sc : 0.f;
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

static WeightHat weight(const F32Args& a) { return WeightHat{a.q, a.ldq, a.s, a.gsize, a.ngroups}; }

hipError_t launch_f32_forward(const F32Args& a, float* Y, hipStream_t st) {
  // Y[t][i] = sum_j X[t][j] W_hat[i][j]
  return run(a.T, a.m, a.k, Mat{a.X, a.k}, WeightHatT{weight(a)}, StoreOut{Y, a.m}, st);
}

hipError_t launch_f32_dx(const F32Args& a, float* dX, hipStream_t st) {
  // dX[t][j] = sum_i dY[t][i] W_hat[i][j]
  return run(a.T, a.k, a.m, Mat{a.dY, a.m}, weight(a), StoreOut{dX, a.k}, st);
}

hipError_t launch_f32_dw(const F32Args& a, float* dA, float* dB, int accumulate, hipStream_t st) {
  // G[i][j] = s M sum_t dY[t][i] X[t][j]
  hipError_t e = run(a.m, a.k, a.T, MatT{a.dY, a.m}, Mat{a.X, a.k},
                     StoreG{a.G, a.k, a.mask, a.ldm, a.s, a.gsize, a.ngroups}, st);
  if (e != hipSuccess) return e;
  // dA[i][rho] = c sum_j G[i][j] B[rho][j]
  e = run(a.m, int64_t(a.r), a.k, Mat{a.G, a.k}, MatT{a.B, a.k}, StoreGrad{dA, a.r, a.c, accumulate}, st);
  if (e != hipSuccess) return e;
  // dB[rho][j] = c sum_i A[i][rho] G[i][j]
  return run(int64_t(a.r), a.k, a.m, MatT{a.A, a.r}, Mat{a.G, a.k}, StoreGrad{dB, a.k, a.c, accumulate}, st);
}

}  // namespace lrqat
