// Setup-side initialisation beyond min-max (run once per layer, before training):
//   * L^p-norm range estimation (Section 4 'Baselines' and Appendix B 'PTQ
//     initialization': the range that minimises the L^p norm between quantized
//     and unquantized weights);
//   * LoftQ with one alternating step (Section 3 'Downcasting operator', the
//     ablation of Section 4.2): INT-b Phi0 and adapters A, B whose product
//     (alpha/r) A B is the best rank-r approximation of the fractional part the
//     integer downcast drops, found by randomized subspace iteration.
#include "common.h"
#include "init.h"

namespace lrqat {

// ============================================================================ L^p range search
// One block per (row, group).  The group's weights are staged in LDS; candidate
// j (1..n_grid) has s_j = fl32(fl32(j / n_grid) * amax / hi) and error
// E_j = sum |w - s_j clip(round(w / s_j))|^p (terms in float32, sums in float64).
// The smallest j of the minimal E_j wins; s0 = s_j.
constexpr int LP_THREADS = 256;
constexpr int LP_MAX_GROUP = int(kLpMaxGroup);  // 64 KiB of LDS

__device__ __forceinline__ float abs_pow(float x, float p, int ip) {
  // |x|^p: repeated products for integer p, exp2(p log2 |x|) otherwise
  const float a = fabsf(x);
  if (ip > 0) {
    float r = a;
    for (int i = 1; i < ip; ++i) r *= a;
    return r;
  }
  return a > 0.f ? exp2f(p * log2f(a)) : 0.f;
}

__global__ __launch_bounds__(LP_THREADS) void k_lp_search(const float* __restrict__ W0, int64_t k, int64_t gsize,
                                                          int ngroups, int bits, float p, int ip, int n_grid,
                                                          float* __restrict__ s0, int32_t* __restrict__ jbest_out) {
  __shared__ float w[LP_MAX_GROUP];
  __shared__ double red[LP_THREADS / 64];
  __shared__ float amax_s;
  const int64_t row = blockIdx.x / ngroups;
  const int grp = int(blockIdx.x % ngroups);
  const float* src = W0 + row * k + int64_t(grp) * gsize;
  const int n = int(gsize);
  float amax = 0.f;
  for (int j = threadIdx.x; j < n; j += LP_THREADS) {
    const float v = src[j];
    w[j] = v;
    amax = fmaxf(amax, fabsf(v));
  }
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = double(amax);
  __syncthreads();
  if (threadIdx.x == 0) amax_s = float(fmax(fmax(red[0], red[1]), fmax(red[2], red[3])));
  __syncthreads();
  amax = amax_s;
  const int lo = -(1 << (bits - 1)), hi = (1 << (bits - 1)) - 1;
  double best = 0.0;
  int jb = 0;
  for (int jj = 1; jj <= n_grid; ++jj) {
    const float sj = amax > 0.f ? (float(jj) / float(n_grid)) * amax / float(hi) : 1.f;
    double e = 0.0;
    for (int j = threadIdx.x; j < n; j += LP_THREADS) {
      const float v = w[j];
      const float q = fminf(fmaxf(__builtin_rintf(v / sj), float(lo)), float(hi));
      e += double(abs_pow(__builtin_fmaf(-sj, q, v), p, ip));
    }
    for (int off = 32; off > 0; off >>= 1) e += __shfl_xor(e, off);
    __syncthreads();  // red reused
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = e;
    __syncthreads();
    const double tot = (red[0] + red[1]) + (red[2] + red[3]);
    if (jj == 1 || tot < best) {
      best = tot;
      jb = jj;
    }
  }
  if (threadIdx.x == 0) {
    const float sj = amax > 0.f ? (float(jb) / float(n_grid)) * amax / float(hi) : 1.f;
    s0[row * ngroups + grp] = sj;
    if (jbest_out) jbest_out[row * ngroups + grp] = jb;
  }
}

hipError_t launch_lp_search(const float* W0, int64_t m, int64_t k, int64_t gsize, int bits, float p, int n_grid,
                            float* s0, int32_t* jbest, hipStream_t st) {
  const int ngroups = int(k / gsize);
  const int ip = (p == float(int(p)) && p >= 1.f && p <= 8.f) ? int(p) : 0;
  k_lp_search<<<unsigned(m * ngroups), LP_THREADS, 0, st>>>(W0, k, gsize, ngroups, bits, p, ip, n_grid, s0, jbest);
  return hipGetLastError();
}

// ============================================================================ LoftQ (T = 1)
// x = fl32(W0 / s0), Phi0 = clip(round(x)) packed INT-b, and the residual
// R = x - Phi0 (|R| <= 1/2 inside the grid), float32 [m][k].  One thread per byte.
__global__ __launch_bounds__(256) void k_loftq_residual(const float* __restrict__ W0, const float* __restrict__ s0,
                                                        int64_t m, int64_t k, int64_t gsize, int ngroups, int bits,
                                                        float* __restrict__ R, uint8_t* __restrict__ phi0) {
  const int lo = -(1 << (bits - 1)), hi = (1 << (bits - 1)) - 1;
  const int64_t per_row = k / 2;
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= m * per_row) return;
  const int64_t row = idx / per_row, col = idx % per_row;
  int v[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int64_t j = 2 * col + e;
    const float x = W0[row * k + j] / s0[row * ngroups + j / gsize];
    v[e] = min(max(int(__builtin_rintf(x)), lo), hi);
    R[row * k + j] = x - float(v[e]);
  }
  phi0[row * per_row + col] = uint8_t((v[0] & 15) | ((v[1] & 15) << 4));
}

// Standard normals for the start block of the subspace iteration: splitmix64
// of (seed + (i + 1) * golden) per index, Box-Muller on consecutive pairs.
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
__global__ __launch_bounds__(256) void k_gauss(float* __restrict__ Z, int64_t n, uint64_t seed) {
  const int64_t pair = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (2 * pair >= n) return;
  const double u1 = 1.0 - double(mix64(seed + uint64_t(2 * pair + 1) * 0x9E3779B97F4A7C15ull) >> 11) * 0x1p-53;
  const double u2 = double(mix64(seed + uint64_t(2 * pair + 2) * 0x9E3779B97F4A7C15ull) >> 11) * 0x1p-53;
  const double rad = sqrt(-2.0 * log(u1));
  const double ang = 6.283185307179586 * u2;
  Z[2 * pair] = float(rad * cos(ang));
  if (2 * pair + 1 < n) Z[2 * pair + 1] = float(rad * sin(ang));
}

// Tall-skinny products with R [m][k]: out_part[chunk][p][c] = sum over t in the
// chunk of X(p, t) V[t][c], X = R (TR = false: p a row, t a column) or R^T
// (TR = true: p a column, t a row); V [T][l], l <= 64.  A block takes 64 values
// of p and one chunk of t, in steps of 64 staged in LDS.
constexpr int TS = 64;
template <bool TR>
__global__ __launch_bounds__(256) void k_tsmm(const float* __restrict__ R, int64_t m, int64_t k,
                                              const float* __restrict__ V, int l, float* __restrict__ part,
                                              int64_t tchunk) {
  // the 64 x 64 block of X: TR as rt[t][p] (pitch 68, 16-byte reads along p), else as rt[p][t]
  // (pitch 65: the rows of R as they lie in memory, conflict-free column reads)
  __shared__ __attribute__((aligned(16))) float rt[TS * 68];
  __shared__ __attribute__((aligned(16))) float vt[TS][64];  // vt[t][c]
  const int64_t P = TR ? k : m, T = TR ? m : k;
  const int64_t p0 = int64_t(blockIdx.x) * TS;
  const int64_t t_begin = int64_t(blockIdx.y) * tchunk, t_end = min(T, t_begin + tchunk);
  // the thread's 4 x 4 register tile: rows p0 + 4 tp .. +3, columns 4 tc .. +3
  const int tp = threadIdx.x & 15, tc = threadIdx.x >> 4;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  for (int64_t t0 = t_begin; t0 < t_end; t0 += TS) {
    // stage the block of R (reads along its contiguous index) and the 64 rows of V
    for (int e = threadIdx.x; e < TS * TS; e += 256) {
      const int a = e >> 6, b = e & 63;
      if (TR) {  // X(p, t) = R[t][p]: a = t, b = p
        const int64_t ri = t0 + a, rj = p0 + b;
        rt[a * 68 + b] = (ri < t_end && rj < k) ? R[ri * k + rj] : 0.f;
      } else {   // X(p, t) = R[p][t]: a = p, b = t
        const int64_t ri = p0 + a, rj = t0 + b;
        rt[a * 65 + b] = (ri < m && rj < t_end) ? R[ri * k + rj] : 0.f;
      }
    }
    for (int e = threadIdx.x; e < TS * 64; e += 256) {
      const int a = e >> 6, c = e & 63;
      vt[a][c] = (t0 + a < t_end && c < l) ? V[(t0 + a) * l + c] : 0.f;
    }
    __syncthreads();
#pragma unroll 4
    for (int t = 0; t < TS; ++t) {
      float x[4];
      if (TR) {
        const f32x4 xv = *reinterpret_cast<const f32x4*>(&rt[t * 68 + 4 * tp]);
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = xv[i];
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = rt[(4 * tp + i) * 65 + t];
      }
      const f32x4 y = *reinterpret_cast<const f32x4*>(&vt[t][4 * tc]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fmaf(x[i], y[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t pp = p0 + 4 * tp + i;
    if (pp < P) {
      float* dst = part + (int64_t(blockIdx.y) * P + pp) * l;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (4 * tc + j < l) dst[4 * tc + j] = acc[i][j];
    }
  }
}

// out[i] = sum over chunks of part[chunk][i], in chunk order.
__global__ __launch_bounds__(256) void k_sum_chunks(const float* __restrict__ part, int64_t nchunks, int64_t n,
                                                    float* __restrict__ out) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int64_t c = 0; c < nchunks; ++c) s += part[c * n + i];
  out[i] = s;
}

// Gram partials: gpart[block][a][b] = sum over the block's rows of Y[row][a] Y[row][b] (float64).
constexpr int GR_ROWS = 256;
__global__ __launch_bounds__(256) void k_gram_part(const float* __restrict__ Y, int64_t P, int l,
                                                   double* __restrict__ gpart) {
  __shared__ float ys[32][64];
  const int64_t r0 = int64_t(blockIdx.x) * GR_ROWS;
  double acc[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) acc[q] = 0.0;
  for (int64_t rb = r0; rb < min(P, r0 + GR_ROWS); rb += 32) {
    for (int e = threadIdx.x; e < 32 * 64; e += 256) {
      const int a = e >> 6, c = e & 63;
      ys[a][c] = (rb + a < P && c < l) ? Y[(rb + a) * l + c] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int pair = threadIdx.x + 256 * q;  // (a, b) = (pair / 64, pair % 64)
      const int a = pair >> 6, b = pair & 63;
      for (int t = 0; t < 32; ++t) acc[q] = __builtin_fma(double(ys[t][a]), double(ys[t][b]), acc[q]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int pair = threadIdx.x + 256 * q;
    const int a = pair >> 6, b = pair & 63;
    if (a < l && b < l) gpart[(int64_t(blockIdx.x) * l + a) * l + b] = acc[q];
  }
}

// One block: G = sum of the Gram partials; L = cholesky(G + eps tr(G) I); M = L^{-T} (float).
// The factorisation is right-looking, one column per step with the trailing update spread over
// the block; the inverse solves L X = I with one thread per column of X.
__global__ __launch_bounds__(256) void k_chol_inv(const double* __restrict__ gpart, int64_t nparts, int l,
                                                  float* __restrict__ M) {
  __shared__ double G[64][65];
  __shared__ double Li[64][65];
  __shared__ double shift_s;
  for (int e = threadIdx.x; e < l * l; e += 256) {
    const int a = e / l, b = e % l;
    double s0 = 0.0, s1 = 0.0;
    int64_t q = 0;
    for (; q + 2 <= nparts; q += 2) {
      s0 += gpart[q * l * l + e];
      s1 += gpart[(q + 1) * l * l + e];
    }
    if (q < nparts) s0 += gpart[q * l * l + e];
    G[a][b] = s0 + s1;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double tr = 0.0;
    for (int a = 0; a < l; ++a) tr += G[a][a];
    shift_s = tr > 0.0 ? 1e-13 * tr : 1e-300;
  }
  __syncthreads();
  if (threadIdx.x < l) G[threadIdx.x][threadIdx.x] += shift_s;
  __syncthreads();
  // lower triangle of G becomes L
  for (int j = 0; j < l; ++j) {
    if (threadIdx.x == 0) {
      const double d = G[j][j];
      G[j][j] = d > 0.0 ? __builtin_sqrt(d) : 1e-150;
    }
    __syncthreads();
    const double dj = G[j][j];
    for (int i = j + 1 + int(threadIdx.x); i < l; i += 256) G[i][j] /= dj;
    __syncthreads();
    // trailing update of the lower triangle: G[i][q] -= L[i][j] L[q][j], j < q <= i
    const int nt = l - j - 1;
    for (int e = threadIdx.x; e < nt * nt; e += 256) {
      const int i = j + 1 + e / nt, q = j + 1 + e % nt;
      if (q <= i) G[i][q] -= G[i][j] * G[q][j];
    }
    __syncthreads();
  }
  // Li = L^{-1}: column jc of Li by forward substitution, one thread per column
  if (int(threadIdx.x) < l) {
    const int jc = threadIdx.x;
    for (int i = 0; i < l; ++i) {
      if (i < jc) {
        Li[i][jc] = 0.0;
        continue;
      }
      double v = i == jc ? 1.0 : 0.0;
      for (int q = jc; q < i; ++q) v -= G[i][q] * Li[q][jc];
      Li[i][jc] = v / G[i][i];
    }
  }
  __syncthreads();
  // M = L^{-T}: M[a][b] = Li[b][a]
  for (int e = threadIdx.x; e < l * l; e += 256) M[e] = float(Li[e % l][e / l]);
}

// Y[row][:] <- Y[row][:] M (l x l), one thread per row, the row in registers (l <= 64).
__global__ __launch_bounds__(256) void k_apply(float* __restrict__ Y, int64_t P, int l, const float* __restrict__ M) {
  __shared__ float Ms[64][64];
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int a = e >> 6, b = e & 63;
    Ms[a][b] = (a < l && b < l) ? M[a * l + b] : 0.f;
  }
  __syncthreads();
  const int64_t row = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (row >= P) return;
  float y[64];
#pragma unroll
  for (int a = 0; a < 64; ++a) y[a] = a < l ? Y[row * l + a] : 0.f;
  for (int b = 0; b < l; ++b) {
    float s = 0.f;
#pragma unroll
    for (int a = 0; a < 64; ++a) s = __builtin_fmaf(y[a], Ms[a][b], s);
    Y[row * l + b] = s;
  }
}

// One block: eigen-decomposition of the symmetric l x l G (sum of the Gram
// partials) by parallel cyclic Jacobi (round-robin pairing, disjoint rotations
// per round), eigenvalues descending; then, with sigma_i = sqrt(lambda_i) and
// the leading r eigenvectors U_r, M1 = U_r sigma^(1/2) / sqrt(c) and
// M2 = U_r sigma^(-1/2) / sqrt(c) (columns with sigma = 0 are zero).
__global__ __launch_bounds__(256) void k_eig_factors(const double* __restrict__ gpart, int64_t nparts, int l, int r,
                                                     double c, float* __restrict__ M1, float* __restrict__ M2,
                                                     float* __restrict__ sigma_out) {
  __shared__ double G[64][65];
  __shared__ double V[64][65];
  __shared__ double cs[32][2];
  __shared__ int pr[32][2];
  __shared__ int order[64];
  __shared__ double off_s;
  const int n = l + (l & 1);  // even for the pairing; a padding index has no rotation
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int a = e >> 6, b = e & 63;
    double s = 0.0;
    if (a < l && b < l)
      for (int64_t q = 0; q < nparts; ++q) s += gpart[q * l * l + a * l + b];
    G[a][b] = s;
    V[a][b] = a == b ? 1.0 : 0.0;
  }
  __syncthreads();
  for (int sweep = 0; sweep < 30; ++sweep) {
    if (threadIdx.x == 0) {
      double off = 0.0, dia = 0.0;
      for (int a = 0; a < l; ++a)
        for (int b = 0; b < l; ++b) (a == b ? dia : off) += G[a][b] * G[a][b];
      off_s = off <= 1e-28 * dia || dia == 0.0 ? -1.0 : off;
    }
    __syncthreads();
    if (off_s < 0.0) break;
    for (int round = 0; round < n - 1; ++round) {
      // pairs of the round: (0, x) and circle pairs, indices of the circle method
      if (threadIdx.x < n / 2) {
        const int t = threadIdx.x;
        int a, b;
        if (t == 0) { a = n - 1; b = round; }
        else { a = (round + t) % (n - 1); b = (round - t + n - 1) % (n - 1); }
        if (a > b) { const int x = a; a = b; b = x; }
        pr[t][0] = a;
        pr[t][1] = b;
        double cth = 1.0, sth = 0.0;
        if (b < l && G[a][b] != 0.0) {
          const double tau = (G[b][b] - G[a][a]) / (2.0 * G[a][b]);
          const double tn = (tau >= 0.0 ? 1.0 : -1.0) / (__builtin_fabs(tau) + __builtin_sqrt(1.0 + tau * tau));
          cth = 1.0 / __builtin_sqrt(1.0 + tn * tn);
          sth = tn * cth;
        }
        cs[t][0] = cth;
        cs[t][1] = sth;
      }
      __syncthreads();
      // rows: G <- J^T G
      for (int e = threadIdx.x; e < (n / 2) * l; e += 256) {
        const int t = e / l, col = e % l;
        const int a = pr[t][0], b = pr[t][1];
        if (b >= l) continue;
        const double cth = cs[t][0], sth = cs[t][1];
        const double ga = G[a][col], gb = G[b][col];
        G[a][col] = cth * ga - sth * gb;
        G[b][col] = sth * ga + cth * gb;
      }
      __syncthreads();
      // columns: G <- G J, V <- V J
      for (int e = threadIdx.x; e < (n / 2) * l; e += 256) {
        const int t = e / l, row = e % l;
        const int a = pr[t][0], b = pr[t][1];
        if (b >= l) continue;
        const double cth = cs[t][0], sth = cs[t][1];
        const double ga = G[row][a], gb = G[row][b];
        G[row][a] = cth * ga - sth * gb;
        G[row][b] = sth * ga + cth * gb;
        const double va = V[row][a], vb = V[row][b];
        V[row][a] = cth * va - sth * vb;
        V[row][b] = sth * va + cth * vb;
      }
      __syncthreads();
    }
  }
  if (threadIdx.x == 0) {
    for (int a = 0; a < l; ++a) order[a] = a;
    for (int a = 0; a < l; ++a) {  // selection sort, descending eigenvalues
      int best = a;
      for (int b = a + 1; b < l; ++b)
        if (G[order[b]][order[b]] > G[order[best]][order[best]]) best = b;
      const int x = order[a]; order[a] = order[best]; order[best] = x;
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < l * r; e += 256) {
    const int a = e / r, j = e % r;
    const int col = order[j];
    const double lam = G[col][col];
    const double sg = lam > 0.0 ? __builtin_sqrt(lam) : 0.0;
    const double rs = __builtin_sqrt(sg);
    const double ic = 1.0 / __builtin_sqrt(c);
    M1[e] = float(V[a][col] * rs * ic);
    M2[e] = float(sg > 0.0 ? V[a][col] / rs * ic : 0.0);
    if (a == 0 && sigma_out) sigma_out[j] = float(sg);
  }
}

// out = Y M (P x l times l x r); transposed: out[j][row] (r x P), else out[row][j].
__global__ __launch_bounds__(256) void k_project(const float* __restrict__ Y, int64_t P, int l,
                                                 const float* __restrict__ M, int r, float* __restrict__ out,
                                                 int transposed) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= P * r) return;
  const int64_t row = transposed ? idx % P : idx / r;
  const int j = int(transposed ? idx / P : idx % r);
  float s = 0.f;
  for (int a = 0; a < l; ++a) s = __builtin_fmaf(Y[row * l + a], M[a * r + j], s);
  out[transposed ? int64_t(j) * P + row : row * r + j] = s;
}

size_t loftq_workspace(int64_t m, int64_t k, int l) {
  auto up = [](size_t b) { return (b + 255) / 256 * 256; };
  const int64_t nt = 16;
  const size_t part = size_t(nt) * size_t(m > k ? m : k) * l * 4;
  const size_t gp = size_t(((m > k ? m : k) + GR_ROWS - 1) / GR_ROWS) * l * l * 8;
  return up(size_t(m) * k * 4) + up(size_t(m) * l * 4) + up(size_t(k) * l * 4) + up(part) + up(gp) +
         up(size_t(l) * l * 4) + 2 * up(size_t(l) * 64 * 4) + up(64 * 4);
}

hipError_t launch_loftq(const float* W0, const float* s0, int64_t m, int64_t k, int64_t gsize, int bits, int r,
                        int l, double c, int n_iter, uint8_t* phi0, float* A, float* B, float* sigma, void* ws,
                        hipStream_t st) {
  auto up = [](size_t b) { return (b + 255) / 256 * 256; };
  const int64_t nt = 16;
  uint8_t* p = static_cast<uint8_t*>(ws);
  float* R = reinterpret_cast<float*>(p); p += up(size_t(m) * k * 4);
  float* Y = reinterpret_cast<float*>(p); p += up(size_t(m) * l * 4);
  float* Z = reinterpret_cast<float*>(p); p += up(size_t(k) * l * 4);
  float* part = reinterpret_cast<float*>(p); p += up(size_t(nt) * size_t(m > k ? m : k) * l * 4);
  double* gpart = reinterpret_cast<double*>(p); p += up(size_t(((m > k ? m : k) + GR_ROWS - 1) / GR_ROWS) * l * l * 8);
  float* M = reinterpret_cast<float*>(p); p += up(size_t(l) * l * 4);
  float* M1 = reinterpret_cast<float*>(p); p += up(size_t(l) * 64 * 4);
  float* M2 = reinterpret_cast<float*>(p);
  const int ngroups = int(k / gsize);
  hipError_t e;
#define LRQAT_CHK(x) do { x; if ((e = hipGetLastError()) != hipSuccess) return e; } while (0)
  LRQAT_CHK((k_loftq_residual<<<unsigned((m * (k / 2) + 255) / 256), 256, 0, st>>>(W0, s0, m, k, gsize, ngroups, bits, R, phi0)));
  LRQAT_CHK((k_gauss<<<unsigned((k * l / 2 + 256) / 256), 256, 0, st>>>(Z, k * l, 0x2406063850ull)));
  // out[P][l] = X V for X = R (P = m) or R^T (P = k)
  auto tsmm = [&](bool tr, const float* V, float* out) -> hipError_t {
    const int64_t P = tr ? k : m, T = tr ? m : k;
    const int64_t tchunk = ((T + nt - 1) / nt + TS - 1) / TS * TS;
    const unsigned ny = unsigned((T + tchunk - 1) / tchunk);
    dim3 grid(unsigned((P + TS - 1) / TS), ny);
    if (tr) k_tsmm<true><<<grid, 256, 0, st>>>(R, m, k, V, l, part, tchunk);
    else k_tsmm<false><<<grid, 256, 0, st>>>(R, m, k, V, l, part, tchunk);
    hipError_t e2 = hipGetLastError();
    if (e2 != hipSuccess) return e2;
    k_sum_chunks<<<unsigned((P * l + 255) / 256), 256, 0, st>>>(part, ny, P * l, out);
    return hipGetLastError();
  };
  // orthonormal columns of Y [P][l] by CholeskyQR, twice
  auto orth = [&](float* Yv, int64_t P) -> hipError_t {
    const unsigned nb = unsigned((P + GR_ROWS - 1) / GR_ROWS);
    for (int pass = 0; pass < 2; ++pass) {
      k_gram_part<<<nb, 256, 0, st>>>(Yv, P, l, gpart);
      k_chol_inv<<<1, 256, 0, st>>>(gpart, nb, l, M);
      k_apply<<<unsigned((P + 255) / 256), 256, 0, st>>>(Yv, P, l, M);
      hipError_t e2 = hipGetLastError();
      if (e2 != hipSuccess) return e2;
    }
    return hipSuccess;
  };
  if ((e = tsmm(false, Z, Y)) != hipSuccess) return e;      // Y = R Z
  for (int it = 0; it < n_iter; ++it) {
    if ((e = orth(Y, m)) != hipSuccess) return e;
    if ((e = tsmm(true, Y, Z)) != hipSuccess) return e;     // Z = R^T Q
    if ((e = orth(Z, k)) != hipSuccess) return e;
    if ((e = tsmm(false, Z, Y)) != hipSuccess) return e;    // Y = R Z
  }
  if ((e = orth(Y, m)) != hipSuccess) return e;             // Q
  if ((e = tsmm(true, Y, Z)) != hipSuccess) return e;       // Zt = R^T Q
  const unsigned nbz = unsigned((k + GR_ROWS - 1) / GR_ROWS);
  LRQAT_CHK((k_gram_part<<<nbz, 256, 0, st>>>(Z, k, l, gpart)));   // Zt^T Zt = (Q^T R)(R^T Q)
  LRQAT_CHK((k_eig_factors<<<1, 256, 0, st>>>(gpart, nbz, l, r, c, M1, M2, sigma)));
  LRQAT_CHK((k_project<<<unsigned((m * r + 255) / 256), 256, 0, st>>>(Y, m, l, M1, r, A, 0)));  // A = Q M1
  LRQAT_CHK((k_project<<<unsigned((k * r + 255) / 256), 256, 0, st>>>(Z, k, l, M2, r, B, 1)));  // B = (Zt M2)^T
#undef LRQAT_CHK
  return hipSuccess;
}

}  // namespace lrqat
