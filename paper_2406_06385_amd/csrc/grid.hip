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
// Tile 64 rows x 128 columns per block of 8 waves; wave w covers the 32x32
// block at rows 32*(w/4), columns 32*(w%4).  delta = c A B is an MFMA
// product of bfloat16 hi/lo splits, A B ~ Ahi Bhi + Ahi Blo + Alo Bhi,
// accumulated in float32.  Its error is below 3*2^-16 sum_rho |A||B| plus the
// float32 accumulation, bounded here by 2^-13 |c| ||A_i|| max_j ||B_:j||
// (Cauchy-Schwarz) <= 2^-13 |c| r max|A_i:| max|B_:j|.  An element whose pre-round value lies within that bound
// of a rounding decision point is decided again from a float64 delta, so the
// grid equals the exact one except within float64 rounding of a .5 point.
//
// The product is formed transposed (B columns as the MFMA row operand), so a
// lane owns one weight row and the columns 8 g + 4 (lane / 32) + e
// (g, e = 0..3) of its wave's block: its Phi0 codes come as one 32-bit (Q8)
// or 16-bit (packed) LDS read per 4 elements, its q nibbles pack in
// registers, and the transposed clip mask is one wave ballot per column pair.
// The pass is latency-bound (one short dependent chain per block), so the
// per-lane state is kept small for occupancy.
constexpr int GR_BM = 64, GR_BN = 128, GR_THREADS = 512;
constexpr int GR_PITCH = 136;  // LDS bytes per staged Phi0 row: 34 dwords keeps the 32 rows of a read on distinct banks

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

// Phi0 code e (0..3) of a 32-bit word of four Q8 bytes or a 16-bit word of four packed nibbles.
template <bool PACKED>
__device__ __forceinline__ int code_of(uint32_t w, int e) {
  if constexpr (PACKED) return int(w << (28 - 4 * e)) >> 28;
  else return int(w << (24 - 8 * e)) >> 24;
}

template <bool PACKED>
__device__ __forceinline__ uint32_t read_codes(const uint8_t* ph, int lr, int lc) {
  if constexpr (PACKED) return *reinterpret_cast<const uint16_t*>(ph + lr * GR_PITCH + (lc >> 1));
  else return *reinterpret_cast<const uint32_t*>(ph + lr * GR_PITCH + lc);
}

// Decision, packing and mask of one block after its Phi0 tile is staged
// (the caller's barrier follows the rank-r product inside).
template <bool PACKED, bool FULL>
__device__ __forceinline__ void grid_body(const GridArgs& a, const uint8_t* ph, int64_t row0, int64_t col0) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  const int wr = 32 * (wave >> 2), wc = 32 * (wave & 3);
  const int lo = -(1 << (a.bits - 1)), hi = (1 << (a.bits - 1)) - 1;
  const int f = PACKED ? 0 : 8 - a.bits;

  // acc[v] = (A B)[row0 + wr + lane % 32][col0 + wc + acc_row(v, lane)]
  f32x16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.f;

  const int64_t arow = row0 + wr + (lane & 31);
  const int64_t bcol = col0 + wc + (lane & 31);
  const bool avec = FULL || ((a.r & 3) == 0 && (reinterpret_cast<uintptr_t>(a.A) & 15) == 0);
  // max |A| over the lane's row and max |B| over its column: ||x|| <= sqrt(r) max|x| bounds the
  // norms, and a zero maximum means an exactly zero delta
  float amax = 0.f, bmax = 0.f;
  for (int r0 = 0; r0 < a.r; r0 += 16) {
    // A operand: A[arow][r0 + 8*half + e]; B operand: B[r0 + 8*half + e][bcol]
    float x[8], y[8];
    const int rb = r0 + 8 * half;
    if (FULL || (avec && arow < a.m && rb + 8 <= a.r)) {
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
    for (int e = 0; e < 8; ++e)
      y[e] = (FULL || (bcol < a.k && rb + e < a.r)) ? a.B[int64_t(rb + e) * a.k + bcol] : 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      amax = fmaxf(amax, fabsf(x[e]));
      bmax = fmaxf(bmax, fabsf(y[e]));
    }
    u32x4 ahi, alo, bhi, blo;
    split8(x, ahi, alo);
    split8(y, bhi, blo);
    acc = mfma32(bhi, ahi, acc);
    acc = mfma32(blo, ahi, acc);
    acc = mfma32(bhi, alo, acc);
  }
  // the two K-halves of every row / column sit in lanes l and l ^ 32; then the max over the 32 columns
  amax = fmaxf(amax, __shfl_xor(amax, 32));
  for (int off = 32; off > 0; off >>= 1) bmax = fmaxf(bmax, __shfl_xor(bmax, off));
  // tau: the error bound of the float32 delta, 2^-13 |c| ||A_i|| max_j ||B_:j|| <= 2^-13 |c| r amax bmax;
  // -1 where delta is exactly zero (a zero A row or all-zero B columns, e.g. B at its zero
  // initialisation), so that no element is re-decided there
  const float tau = (amax == 0.f || bmax == 0.f) ? -1.f : 0x1p-13f * fabsf(a.c) * float(a.r) * amax * bmax;
  __syncthreads();  // Phi0 tile staged

  const int lr = wr + (lane & 31);                            // the lane's row in the tile
  const bool row_ok = FULL || lr < int(min<int64_t>(a.m - row0, GR_BM));
  const int kr = int(min<int64_t>(a.k - col0, GR_BN)) - wc - 4 * half;  // the lane's columns 8 g + e < kr are inside
  auto col_of = [&](int v) { return wc + 8 * (v >> 2) + 4 * half + (v & 3); };
  auto inside = [&](int v) { return FULL || (row_ok && 8 * (v >> 2) + (v & 3) < kr); };

  // Rounding decision per element from the float32 delta.
  int ut[16];
  bool need = false;  // some element of the lane lies within tau of a decision point
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const uint32_t w = read_codes<PACKED>(ph, lr, col_of(4 * g));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int v = 4 * g + e;
      float margin;
      ut[v] = grid_round(code_of<PACKED>(w, e), f, a.c * acc[v], &margin);
      need |= margin <= tau && inside(v);
    }
  }
  // float64 re-decision of those elements (rare: the wave takes this branch only if one of its lanes needs it)
  if (__builtin_amdgcn_ballot_w64(need)) {
    const int64_t row = row0 + lr;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int code = code_of<PACKED>(read_codes<PACKED>(ph, lr, col_of(v & 12)), v & 3);
      float margin;
      grid_round(code, f, a.c * acc[v], &margin);
      if (need && margin <= tau && inside(v)) {
        const int64_t col = col0 + col_of(v);
        double d0 = 0.0, d1 = 0.0, d2 = 0.0, d3 = 0.0;  // independent partial sums keep the loads in flight
        int rho = 0;
        for (; rho + 4 <= a.r; rho += 4) {
          d0 = __builtin_fma(double(a.A[row * a.r + rho]), double(a.B[int64_t(rho) * a.k + col]), d0);
          d1 = __builtin_fma(double(a.A[row * a.r + rho + 1]), double(a.B[int64_t(rho + 1) * a.k + col]), d1);
          d2 = __builtin_fma(double(a.A[row * a.r + rho + 2]), double(a.B[int64_t(rho + 2) * a.k + col]), d2);
          d3 = __builtin_fma(double(a.A[row * a.r + rho + 3]), double(a.B[int64_t(rho + 3) * a.k + col]), d3);
        }
        for (; rho < a.r; ++rho) d0 = __builtin_fma(double(a.A[row * a.r + rho]), double(a.B[int64_t(rho) * a.k + col]), d0);
        ut[v] = grid_round_f64(code, f, a.c64 * ((d0 + d1) + (d2 + d3)));
      }
    }
  }

  // Clip to the grid; pack the nibbles (cols 8g + 4 half .. +3 -> 16 bits) and
  // gather the clip-mask bits column by column with wave ballots.
  // Lane L < 32 writes the mask word of column wc + L: the ballot of element v = 4 (L / 8) + L % 4,
  // its low half for L % 8 < 4, else its high half.
  const int myv = 4 * ((lane >> 3) & 3) + (lane & 3);
  uint64_t mbal = 0;
  uint32_t P[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    uint32_t nib = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int v = 4 * g + e;
      const bool ok = inside(v);
      const int q = min(max(ut[v], lo), hi);
      nib |= uint32_t(ok ? q & 15 : 0) << (4 * e);
      // lanes 0..31 of the ballot: column 8 g + e of the block; lanes 32..63: that column + 4
      const uint64_t bal = __builtin_amdgcn_ballot_w64(ok && q == ut[v]);
      mbal = myv == v ? bal : mbal;
    }
    P[g] = nib;
  }
  const uint32_t mword = (lane & 4) ? uint32_t(mbal >> 32) : uint32_t(mbal);

  // Packed q: the 8-column word of group g is half 0's nibbles | half 1's << 16;
  // half 0 stores groups 0-1 and half 1 groups 2-3 (16 columns, 8 bytes each).
  if (row_ok) {  // lanes l and l ^ 32 share the row, so the exchange partner is active
    const int64_t row = row0 + lr;
    const uint32_t send = half ? (P[0] | (P[1] << 16)) : (P[2] | (P[3] << 16));
    const uint32_t recv = __shfl_xor(send, 32);
    uint32_t w0, w1;
    if (half) {
      w0 = (recv & 0xffffu) | (P[2] << 16);
      w1 = (recv >> 16) | (P[3] << 16);
    } else {
      w0 = P[0] | (recv << 16);
      w1 = P[1] | (recv & 0xffff0000u);
    }
    const int64_t c = col0 + wc + 16 * half;                 // first of the 16 columns
    uint8_t* dst = a.qout + row * a.ldq + (c >> 1);
    if (FULL ? (reinterpret_cast<uintptr_t>(dst) & 7) == 0
             : (c + 16 <= a.kq && (reinterpret_cast<uintptr_t>(dst) & 7) == 0)) {
      *reinterpret_cast<u32x2*>(dst) = u32x2{w0, w1};
    } else if (c < a.kq) {
      const int64_t nb = min<int64_t>(8, (a.kq - c + 1) >> 1);
      for (int64_t byte = 0; byte < nb; ++byte) dst[byte] = uint8_t((byte < 4 ? w0 : w1) >> (8 * (byte & 3)));
    }
  }
  // Clip-mask bits, transposed: bit (row % 8) of byte [col][row / 8]; one 32-row word per lane.
  if (a.mout && lane < 32) {
    const int64_t col = col0 + wc + lane;
    if (FULL || col < a.kq) *reinterpret_cast<uint32_t*>(a.mout + col * a.ldm + ((row0 + wr) >> 3)) = mword;
  }
}

template <bool PACKED>
__global__ __launch_bounds__(GR_THREADS) void k_grid(GridArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t ph[GR_BM * GR_PITCH];  // the block's Phi0 bytes
  const int64_t ncb = (a.kq + GR_BN - 1) / GR_BN;
  const int64_t row0 = int64_t(blockIdx.x / ncb) * GR_BM;
  const int64_t col0 = int64_t(blockIdx.x % ncb) * GR_BN;

  // Stage the Phi0 tile in LDS first so its loads overlap the rank-r product.
  // Rows past m read as zeros (buffer range); columns past k are never used.
  {
    constexpr int nbytes = (PACKED ? GR_BN / 2 : GR_BN) / 8;  // per thread: 16 (Q8) or 8 (packed)
    const int64_t cb0 = PACKED ? col0 / 2 : col0;
    const auto r = grid_rsrc(a.phi0 + row0 * a.ld_phi + cb0, (a.m - row0) * a.ld_phi - cb0);
    const int tr = threadIdx.x >> 3, seg = threadIdx.x & 7;   // 8 threads per row
    const int off = int(tr * a.ld_phi) + seg * nbytes;
    uint8_t* dst = ph + tr * GR_PITCH + seg * nbytes;
    if ((a.ld_phi & (nbytes - 1)) == 0) {
      if constexpr (PACKED) {
        *reinterpret_cast<u32x2*>(dst) = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
      } else {
        const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
        *reinterpret_cast<u32x2*>(dst) = u32x2{v[0], v[1]};
        *reinterpret_cast<u32x2*>(dst + 8) = u32x2{v[2], v[3]};
      }
    } else {
      for (int o = 0; o < nbytes; ++o) dst[o] = uint8_t(__builtin_amdgcn_raw_buffer_load_b8(r, off + o, 0, 0));
    }
  }

  // Interior blocks (every row and column inside the matrix, r a multiple of
  // 16) take a variant without bounds checks.
  const bool full = row0 + GR_BM <= a.m && col0 + GR_BN <= a.k && (a.r & 15) == 0 &&
                    (reinterpret_cast<uintptr_t>(a.A) & 15) == 0;
  if (full) grid_body<PACKED, true>(a, ph, row0, col0);
  else grid_body<PACKED, false>(a, ph, row0, col0);
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
  if (a.packed) k_grid<true><<<unsigned(nblocks), GR_THREADS, 0, st>>>(a);
  else k_grid<false><<<unsigned(nblocks), GR_THREADS, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_act_quant(const uint16_t* X, int64_t T, int64_t k, int8_t* n, int64_t ldn, float* sx,
                            hipStream_t st) {
  k_act_quant<<<unsigned(T), 256, 0, st>>>(X, k, n, ldn, sx);
  return hipGetLastError();
}

}  // namespace lrqat
