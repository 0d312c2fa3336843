// Weight-side kernels of the LR-QAT layer:
//   * setup: min-max range estimation and the downcast Phi0 = phi(W0/s0)
//     (Section 3, Eq. phi, Eq. phi_fixed_point);
//   * the integer grid q = clip(round(Phi0 + (alpha/r) A B)) with its STE
//     clip mask (Section 3, Eq. lr_qat), written double-packed -- this is both
//     the per-call reconstruction pass of the forward/backward and the merge
//     for inference (W_Z);
//   * per-token int8 activation quantisation (Section 4, W4A8).
#include "kernels.h"

namespace lrqat {

// ============================================================================ setup

// One block per (row, group): s0 = max|W0[row, group]| / (2^(b-1)-1); 0 -> 1.
__global__ __launch_bounds__(256) void k_minmax_scale(const float* __restrict__ W0, int64_t k,
                                                      int64_t gsize, int ngroups, float hi,
                                                      float* __restrict__ s0) {
  const int64_t row = blockIdx.x / ngroups;
  const int grp = int(blockIdx.x % ngroups);
  const float* p = W0 + row * k + int64_t(grp) * gsize;
  float amax = 0.f;
  for (int64_t j = threadIdx.x; j < gsize; j += blockDim.x) amax = fmaxf(amax, fabsf(p[j]));
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  __shared__ float red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
  __syncthreads();
  if (threadIdx.x == 0) {
    float a = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    s0[row * ngroups + grp] = a > 0.f ? a / hi : 1.f;
  }
}

// Phi0 = phi(W0 / s0).  Q8: one thread per element; packed: one per byte.
__global__ __launch_bounds__(256) void k_encode(const float* __restrict__ W0, const float* __restrict__ s0,
                                                int64_t m, int64_t k, int64_t gsize, int ngroups, int bits,
                                                int packed, void* __restrict__ phi0) {
  const int lo = -(1 << (bits - 1)), hi = (1 << (bits - 1)) - 1;
  const int64_t per_row = packed ? k / 2 : k;
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= m * per_row) return;
  const int64_t row = idx / per_row, col = idx % per_row;
  if (!packed) {
    const float x = W0[row * k + col] / s0[row * ngroups + col / gsize];
    const float xc = fminf(fmaxf(x, float(lo)), float(hi));
    const int f = 8 - bits;
    static_cast<int8_t*>(phi0)[row * k + col] = int8_t(int(__builtin_rintf(xc * float(1 << f))));
  } else {
    int v[2];
    #pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int64_t j = 2 * col + e;
      const float x = W0[row * k + j] / s0[row * ngroups + j / gsize];
      v[e] = min(max(int(__builtin_rintf(x)), lo), hi);
    }
    static_cast<uint8_t*>(phi0)[row * per_row + col] = uint8_t((v[0] & 15) | ((v[1] & 15) << 4));
  }
}

// ============================================================================ grid
// Tile 64 rows x 128 columns per block of 4 waves; wave w covers rows
// 32*(w/2) and columns 64*(w%2) as two 32x32 MFMA blocks.  delta = c A B is
// an MFMA product of bfloat16 hi/lo splits, A B ~ Ahi Bhi + Ahi Blo + Alo Bhi,
// accumulated in float32.  Its error is below 3*2^-16 sum_rho |A||B| plus the
// float32 accumulation, bounded here by 2^-13 |c| max_i ||A_i|| ||B_:j||
// (Cauchy-Schwarz).  An element whose pre-round value lies within that bound
// of a rounding decision point is decided again from a float64 delta, so the
// grid equals the exact one except within float64 rounding of a .5 point.
constexpr int GR_BM = 64, GR_BN = 128;

// 8 consecutive floats -> bf16 hi part and bf16 lo part (x - hi), packed.
__device__ __forceinline__ void split8(const float (&x)[8], u32x4& hi, u32x4& lo) {
  #pragma unroll
  for (int p = 0; p < 4; ++p) {
    const uint32_t h = pack_bf16x2(x[2 * p], x[2 * p + 1]);
    hi[p] = h;
    lo[p] = pack_bf16x2(x[2 * p] - bf16_lo(h), x[2 * p + 1] - bf16_hi(h));
  }
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t grid_rsrc(const void* base, int64_t bytes) {
  const int64_t n = bytes < 0 ? 0 : (bytes > int64_t(0xFFFFFFFF) ? int64_t(0xFFFFFFFF) : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), short(0), int(uint32_t(n)), 0x00020000);
}

__global__ __launch_bounds__(256) void k_grid(GridArgs a) {
  __shared__ uint8_t qs[GR_BM][GR_BN];     // (q & 15) | 0x10 when the element is inside the grid
  __shared__ uint8_t ph[GR_BM][GR_BN];     // the block's Phi0 bytes (GR_BN/2 per row when packed)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t ncb = (a.kq + GR_BN - 1) / GR_BN;
  const int64_t row0 = int64_t(blockIdx.x / ncb) * GR_BM;
  const int64_t col0 = int64_t(blockIdx.x % ncb) * GR_BN;
  const int wr = 32 * (wave >> 1), wc = 64 * (wave & 1);
  const int lo = -(1 << (a.bits - 1)), hi = (1 << (a.bits - 1)) - 1;
  const int f = a.packed ? 0 : 8 - a.bits;

  // Stage the Phi0 tile in LDS first so its loads overlap the rank-r product.
  // Rows past m read as zeros (buffer range); columns past k are never used.
  {
    const int64_t bpr = a.packed ? GR_BN / 2 : GR_BN;          // bytes per tile row
    const int64_t cb0 = a.packed ? col0 / 2 : col0;
    const auto r = grid_rsrc(a.phi0 + row0 * a.ld_phi + cb0, (a.m - row0) * a.ld_phi - cb0);
    const int tr = threadIdx.x >> 2, seg = threadIdx.x & 3;   // 4 threads per row
    const int64_t nbytes = bpr / 4;                            // 32 (fixed point) or 16 (packed)
    if ((a.ld_phi & 15) == 0) {
      for (int64_t o = 0; o < nbytes; o += 16) {
        const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
            r, int(tr * a.ld_phi + seg * nbytes + o), 0, 0));
        *reinterpret_cast<u32x4*>(&ph[tr][seg * nbytes + o]) = v;
      }
    } else {
      for (int64_t o = 0; o < nbytes; ++o)
        ph[tr][seg * nbytes + o] = uint8_t(__builtin_amdgcn_raw_buffer_load_b8(r, int(tr * a.ld_phi + seg * nbytes + o), 0, 0));
    }
  }

  f32x16 acc[2];
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[b][v] = 0.f;

  const int64_t arow = row0 + wr + (lane & 31);
  const int half = lane >> 5;
  const bool avec = (a.r & 3) == 0 && (reinterpret_cast<uintptr_t>(a.A) & 15) == 0;
  float a2 = 0.f, b2[2] = {0.f, 0.f};  // squared norms: the lane's A row, its B columns
  for (int r0 = 0; r0 < a.r; r0 += 16) {
    // A operand: A[arow][r0 + 8*half + e]
    float x[8];
    const int rb = r0 + 8 * half;
    if (avec && arow < a.m && rb + 8 <= a.r) {
      const f32x4 u = *reinterpret_cast<const f32x4*>(a.A + arow * a.r + rb);
      const f32x4 w = *reinterpret_cast<const f32x4*>(a.A + arow * a.r + rb + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = u[e];
        x[4 + e] = w[e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = (arow < a.m && rb + e < a.r) ? a.A[arow * a.r + rb + e] : 0.f;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) a2 += x[e] * x[e];
    u32x4 ahi, alo;
    split8(x, ahi, alo);
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int64_t bcol = col0 + wc + 32 * b + (lane & 31);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        x[e] = (bcol < a.k && rb + e < a.r) ? a.B[int64_t(rb + e) * a.k + bcol] : 0.f;
        b2[b] += x[e] * x[e];
      }
      u32x4 bhi, blo;
      split8(x, bhi, blo);
      acc[b] = mfma32(ahi, bhi, acc[b]);
      acc[b] = mfma32(ahi, blo, acc[b]);
      acc[b] = mfma32(alo, bhi, acc[b]);
    }
  }
  // the two K-halves of every row / column sit in lanes l and l ^ 32
  a2 += __shfl_xor(a2, 32);
  for (int off = 16; off > 0; off >>= 1) a2 = fmaxf(a2, __shfl_xor(a2, off));  // max over the 32 rows
  float tau[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    b2[b] += __shfl_xor(b2[b], 32);
    tau[b] = 0x1p-13f * fabsf(a.c) * sqrtf(a2 * b2[b]);
  }
  __syncthreads();  // Phi0 tile staged

  // Rounding decision per element -> LDS as (q & 15) | (in-range ? 0x10 : 0).
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int lc = wc + 32 * b + (lane & 31);
    const int64_t col = col0 + lc;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int lr = wr + acc_row(v, lane);
      const int64_t row = row0 + lr;
      int code;
      if (a.packed) code = int(uint32_t(ph[lr][lc >> 1]) << (28 - 4 * (lc & 1))) >> 28;
      else code = int(int8_t(ph[lr][lc]));
      float margin;
      int ut = grid_round(code, f, a.c * acc[b][v], &margin);
      if (margin <= tau[b] && row < a.m && col < a.k) {
        // float64 re-decision; independent partial sums keep the loads in flight
        double d0 = 0.0, d1 = 0.0, d2 = 0.0, d3 = 0.0;
        int rho = 0;
        for (; rho + 4 <= a.r; rho += 4) {
          d0 = __builtin_fma(double(a.A[row * a.r + rho]), double(a.B[int64_t(rho) * a.k + col]), d0);
          d1 = __builtin_fma(double(a.A[row * a.r + rho + 1]), double(a.B[int64_t(rho + 1) * a.k + col]), d1);
          d2 = __builtin_fma(double(a.A[row * a.r + rho + 2]), double(a.B[int64_t(rho + 2) * a.k + col]), d2);
          d3 = __builtin_fma(double(a.A[row * a.r + rho + 3]), double(a.B[int64_t(rho + 3) * a.k + col]), d3);
        }
        for (; rho < a.r; ++rho) d0 = __builtin_fma(double(a.A[row * a.r + rho]), double(a.B[int64_t(rho) * a.k + col]), d0);
        ut = grid_round_f64(code, f, a.c64 * ((d0 + d1) + (d2 + d3)));
      }
      const int q = min(max(ut, lo), hi);
      qs[lr][lc] = (row < a.m && col < a.k) ? uint8_t((q & 15) | (q == ut ? 0x10 : 0)) : uint8_t(0);
    }
  }
  __syncthreads();

  // Packed q: row t/4, 32 columns per thread -> 16 bytes.
  {
    const int lr = threadIdx.x >> 2, seg = threadIdx.x & 3;
    const int64_t row = row0 + lr;
    const int64_t cbase = col0 + 32 * seg;          // first column of this segment
    if (row < a.m && cbase < a.kq) {
      uint32_t w[4];
      #pragma unroll
      for (int p = 0; p < 4; ++p) {
        uint32_t acc_w = 0;
        #pragma unroll
        for (int e = 0; e < 8; ++e) acc_w |= uint32_t(qs[lr][32 * seg + 8 * p + e] & 15) << (4 * e);
        w[p] = acc_w;
      }
      uint8_t* dst = a.qout + row * a.ldq + (cbase >> 1);
      if (cbase + 32 <= a.kq && ((reinterpret_cast<uintptr_t>(dst) & 15) == 0)) {
        *reinterpret_cast<u32x4*>(dst) = u32x4{w[0], w[1], w[2], w[3]};
      } else {
        const int64_t nbytes = min<int64_t>(16, (a.kq - cbase + 1) >> 1);
        for (int64_t byte = 0; byte < nbytes; ++byte) dst[byte] = uint8_t(w[byte >> 2] >> (8 * (byte & 3)));
      }
    }
  }
  // Clip-mask bits, transposed: bit (row % 8) of byte [col][row / 8]; one
  // 32-row word per thread (column t % 128, rows 32 (t / 128) .. +31).
  if (a.mout) {
    const int c = threadIdx.x & 127, hr = threadIdx.x >> 7;
    const int64_t col = col0 + c;
    if (col < a.kq) {
      uint32_t bitsw = 0;
#pragma unroll
      for (int e = 0; e < 32; ++e) bitsw |= uint32_t((qs[32 * hr + e][c] >> 4) & 1) << e;
      *reinterpret_cast<uint32_t*>(a.mout + col * a.ldm + ((row0 + 32 * hr) >> 3)) = bitsw;
    }
  }
}

// ============================================================================ activations
// One block per token row: s_x = max|X_t| / 127, n = clip(round(X_t / s_x), -128, 127).
// Columns k..ldn-1 of n are written as 0.
__global__ __launch_bounds__(256) void k_act_quant(const uint16_t* __restrict__ X, int64_t k,
                                                   int8_t* __restrict__ n, int64_t ldn,
                                                   float* __restrict__ sx) {
  const int64_t row = blockIdx.x;
  const uint16_t* x = X + row * k;
  float amax = 0.f;
  for (int64_t j = threadIdx.x; j < k; j += 256) amax = fmaxf(amax, fabsf(bf16_to_f32(x[j])));
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  __shared__ float red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float s = amax / 127.f;
  if (threadIdx.x == 0) sx[row] = s;
  int8_t* out = n + row * ldn;
  for (int64_t j = threadIdx.x; j < ldn; j += 256) {
    int v = 0;
    if (j < k && s > 0.f) v = min(max(int(__builtin_rintf(bf16_to_f32(x[j]) / s)), -128), 127);
    out[j] = int8_t(v);
  }
}

// ============================================================================ launchers

hipError_t launch_minmax_scale(const float* W0, int64_t m, int64_t k, int64_t gsize, int bits, float* s0,
                               hipStream_t st) {
  const int ngroups = int(k / gsize);
  k_minmax_scale<<<unsigned(m * ngroups), 256, 0, st>>>(W0, k, gsize, ngroups,
                                                          float((1 << (bits - 1)) - 1), s0);
  return hipGetLastError();
}

hipError_t launch_encode(const float* W0, const float* s0, int64_t m, int64_t k, int64_t gsize, int bits,
                         int packed, void* phi0, hipStream_t st) {
  const int64_t n = m * (packed ? k / 2 : k);
  const int ngroups = int(k / gsize);
  k_encode<<<unsigned((n + 255) / 256), 256, 0, st>>>(W0, s0, m, k, gsize, ngroups, bits, packed, phi0);
  return hipGetLastError();
}

hipError_t launch_grid(const GridArgs& a, hipStream_t st) {
  const int64_t nblocks = ((a.kq + GR_BN - 1) / GR_BN) * ((a.m + GR_BM - 1) / GR_BM);
  k_grid<<<unsigned(nblocks), 256, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_act_quant(const uint16_t* X, int64_t T, int64_t k, int8_t* n, int64_t ldn, float* sx,
                            hipStream_t st) {
  k_act_quant<<<unsigned(T), 256, 0, st>>>(X, k, n, ldn, sx);
  return hipGetLastError();
}

}  // namespace lrqat
