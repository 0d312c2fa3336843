// Weight-side kernels of the LR-QAT layer:
//   * setup: min-max range estimation and the downcast Phi0 = phi(W0/s0)
//     (Section 3, Eq. phi, Eq. phi_fixed_point);
//   * the integer grid q = clip(round(Phi0 + (alpha/r) A B)) with its STE
//     clip mask (Section 3, Eq. lr_qat), written double-packed -- this is both
//     the per-call reconstruction pass of the forward/backward and the merge
//     for inference (W_Z);
//   * per-token int8 activation quantisation (Section 4, W4A8).
#include "grid_swar.h"
#include "kernels.h"

namespace lrqat {

// ============================================================================ setup

// One block per (row, group): s0 = max|W0[row, group]| / (2^(b-1)-1); 0 -> 1.
// With z0 (asymmetric): the range [min(W, 0), max(W, 0)] onto [lo, hi],
// s0 = (max - min) / (2^b - 1), z0 = clip(lo - round(min / s0), lo, hi);
// a zero range gives s0 = 1, z0 = 0.
__global__ __launch_bounds__(256) void k_minmax_scale(const float* __restrict__ W0, int64_t k,
                                                      int64_t gsize, int ngroups, int bits,
                                                      float* __restrict__ s0, int32_t* __restrict__ z0) {
  const int64_t row = blockIdx.x / ngroups;
  const int grp = int(blockIdx.x % ngroups);
  const float* p = W0 + row * k + int64_t(grp) * gsize;
  float amax = 0.f, vmin = 0.f, vmax = 0.f;
  for (int64_t j = threadIdx.x; j < gsize; j += blockDim.x) {
    const float v = p[j];
    amax = fmaxf(amax, fabsf(v));
    vmin = fminf(vmin, v);
    vmax = fmaxf(vmax, v);
  }
  for (int off = 32; off > 0; off >>= 1) {
    amax = fmaxf(amax, __shfl_xor(amax, off));
    vmin = fminf(vmin, __shfl_xor(vmin, off));
    vmax = fmaxf(vmax, __shfl_xor(vmax, off));
  }
  __shared__ float red[3][4];
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = amax;
    red[1][threadIdx.x >> 6] = vmin;
    red[2][threadIdx.x >> 6] = vmax;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int lo = -(1 << (bits - 1)), hi = (1 << (bits - 1)) - 1;
    const int64_t at = row * ngroups + grp;
    if (!z0) {
      const float a = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
      s0[at] = a > 0.f ? a / float(hi) : 1.f;
    } else {
      const float mn = fminf(fminf(red[1][0], red[1][1]), fminf(red[1][2], red[1][3]));
      const float mx = fmaxf(fmaxf(red[2][0], red[2][1]), fmaxf(red[2][2], red[2][3]));
      const float range = mx - mn;
      if (range > 0.f) {
        const float s = range / float((1 << bits) - 1);
        s0[at] = s;
        z0[at] = min(max(lo - int(__builtin_rintf(mn / s)), lo), hi);
      } else {
        s0[at] = 1.f;
        z0[at] = 0;
      }
    }
  }
}

// Phi0 = phi(W0 / s0 + z0).  Q8: one thread per element; packed: one per byte.
// The zero offset is added outside the rounding: clip(round(2^f x) + 2^f z)
// (fixed point), clip(round(x) + z) (INT-b); without z, round(2^f clip(x)).
__global__ __launch_bounds__(256) void k_encode(const float* __restrict__ W0, const float* __restrict__ s0,
                                                const int32_t* __restrict__ z0, int64_t m, int64_t k,
                                                int64_t gsize, int ngroups, int bits, int packed,
                                                void* __restrict__ phi0) {
  const int lo = -(1 << (bits - 1)), hi = (1 << (bits - 1)) - 1;
  const int64_t per_row = packed ? k / 2 : k;
  const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= m * per_row) return;
  const int64_t row = idx / per_row, col = idx % per_row;
  if (!packed) {
    const int64_t gi = row * ngroups + col / gsize;
    const float x = W0[row * k + col] / s0[gi];
    const int f = 8 - bits;
    int code;
    if (z0) {
      code = min(max(int(__builtin_rintf(x * float(1 << f))) + z0[gi] * (1 << f), lo * (1 << f)), hi * (1 << f));
    } else {
      const float xc = fminf(fmaxf(x, float(lo)), float(hi));
      code = int(__builtin_rintf(xc * float(1 << f)));
    }
    static_cast<int8_t*>(phi0)[row * k + col] = int8_t(code);
  } else {
    int v[2];
    #pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int64_t j = 2 * col + e;
      const int64_t gi = row * ngroups + j / gsize;
      const float x = W0[row * k + j] / s0[gi];
      v[e] = min(max(int(__builtin_rintf(x)) + (z0 ? z0[gi] : 0), lo), hi);
    }
    static_cast<uint8_t*>(phi0)[row * per_row + col] = uint8_t((v[0] & 15) | ((v[1] & 15) << 4));
  }
}

// ============================================================================ grid
// A block owns 256 adjacent columns and nit consecutive 16-row blocks; wave w
// takes columns 64 w .. 64 w + 63 of the block and walks its nit row blocks
// (prefetching the next one).  For a 16 x 64 wave tile, delta = c A B comes
// from 16x16x32 MFMAs on bfloat16 hi/lo splits,
// A B ~ Ahi Bhi + Ahi Blo + Alo Bhi, accumulated in float32.  The product is
// transposed (B columns are the MFMA row operand) and the B columns of column
// block cb (0..3) are permuted: MFMA row i stands for column
// 16 (i / 4) + 4 cb + i % 4, so lane l owns weight row l % 16 and the 16
// consecutive columns 16 (l / 16) .. +15 of the tile.  Its Phi0 codes are one
// 16-byte (Q8) or 8-byte (packed) load, its q nibbles one 8-byte store (16
// bytes for grids wider than 4 bits), and its clip-mask bits one 16-bit store.
//
// Error bound of the float32 delta: the split drops terms below
// 3.0001 * 2^-16 |a||b| per product; float32 accumulation of the 3r products
// and the scaling by c add at most (3r + 2) 2^-23 sum |products| -- one unit
// in the last place per addition, which also covers an accumulator that
// truncates instead of rounding to nearest (the MFMA's internal rounding is
// not specified).  With Cauchy-Schwarz, sum_rho |A_i,rho||B_rho,j| <=
// ||A_i:|| ||B_:j||, so |delta32 - delta| <= tau_coef * ||A_i:|| *
// max_j ||B_:j||, where tau_coef = 1.02 (3 * 2^-16 + (3r + 2) 2^-23) |c|
// (the 1.02 covers the float32 norms).
// Near a decision point n != 0 the float32 sum u - n adds at most 2^-23 |n|;
// near n = 0 it is exact.  Elements inside that bound are decided again from
// a float64 delta, so the grid equals the exact one except within float64
// rounding of a .5 point.
#ifndef LRQAT_GRW_MIN_BLOCKS
#define LRQAT_GRW_MIN_BLOCKS 512
#endif
constexpr int GR_COLS = 64, GR_THREADS = 256, GR_MIN_BLOCKS = 512, GRW_MIN_BLOCKS = LRQAT_GRW_MIN_BLOCKS;

// 16x16x32 MFMA, D(16x16, f32) += P(16x32, bf16) Q(32x16, bf16): lane l
// supplies row l % 16 of P and column l % 16 of Q, each with the 8 K-values
// 8 (l / 16) .. +7; D element v of lane l is D[4 (l / 16) + v][l % 16].
__device__ __forceinline__ f32x4 mfma16(const u32x4& p, const u32x4& q, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, p), __builtin_bit_cast(bf16x8, q), c, 0, 0,
                                                 0);
}

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
__device__ __forceinline__ float gld(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, int(off), 0, 0));
}

// Upper bound of the Euclidean norm from a float32 sum of squares and the
// exact max |x| (sqrt(n) max|x| where the squares may have underflowed).
__device__ __forceinline__ float norm_bound(float ssq, float amax, int n) {
  return ssq > 0x1p-100f ? __builtin_sqrtf(ssq) : __builtin_sqrtf(float(n)) * amax;
}

// The lane's 16 Phi0 codes (columns 16 (l / 16) .. +15 of the tile): four
// 32-bit words of Q8 bytes, or two words of packed nibbles.
struct PhiRegs {
  uint32_t w[4];
};

// Buffer resources take a wave-uniform base (here the first row of the wave's
// 16-row block); rows past m read as zeros.
template <bool PACKED>
__device__ __forceinline__ void load_phi(PhiRegs& P, const GridArgs& a, int64_t rowblk, int64_t col0, bool vec) {
  const int lane = threadIdx.x & 63;
  const int nb = PACKED ? 8 : 16;
  const int64_t row0 = rowblk * 16, cb0 = PACKED ? col0 / 2 : col0;
  const auto r = grid_rsrc(a.phi0 + row0 * a.ld_phi + cb0, (a.m - row0) * a.ld_phi - cb0);
  const uint32_t off = uint32_t((lane & 15) * a.ld_phi + nb * (lane >> 4));
  if (vec) {
    if constexpr (PACKED) {
      const u32x2 v = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, int(off), 0, 0));
      P.w[0] = v[0];
      P.w[1] = v[1];
      P.w[2] = P.w[3] = 0u;
    } else {
      const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, int(off), 0, 0));
#pragma unroll
      for (int q = 0; q < 4; ++q) P.w[q] = v[q];
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) P.w[q] = 0u;
    for (int b = 0; b < nb; ++b)
      P.w[b >> 2] |= uint32_t(__builtin_amdgcn_raw_buffer_load_b8(r, int(off + b), 0, 0)) << (8 * (b & 3));
  }
}

// Code of column 16 (l / 16) + idx (idx = 4 cb + v) of the lane.
template <bool PACKED>
__device__ __forceinline__ int phi_code(const PhiRegs& P, int idx) {
  if constexpr (PACKED) return int(P.w[idx >> 3] << (28 - 4 * (idx & 7))) >> 28;
  else return int(P.w[idx >> 2] << (24 - 8 * (idx & 3))) >> 24;
}

// The same with a run-time index (the rare float64 path).
template <bool PACKED>
__device__ __forceinline__ int phi_code_dyn(const PhiRegs& P, int idx) {
  const int wi = PACKED ? idx >> 3 : idx >> 2;
  const uint32_t w = wi == 0 ? P.w[0] : wi == 1 ? P.w[1] : wi == 2 ? P.w[2] : P.w[3];
  if constexpr (PACKED) return int(w << (28 - 4 * (idx & 7))) >> 28;
  else return int(w << (24 - 8 * (idx & 3))) >> 24;
}

// A operand of one K-step: A[row][32 ks + 8 (l / 16) .. +7] of the lane's
// row (zero past r or m).
__device__ __forceinline__ void load_a(float (&x)[8], const GridArgs& a, int64_t rowblk, int ks, bool avec) {
  const int lane = threadIdx.x & 63;
  const int rb = 32 * ks + 8 * (lane >> 4);
  const int64_t row0 = rowblk * 16;
  const auto r = grid_rsrc(a.A + row0 * a.r, (a.m - row0) * int64_t(a.r) * 4);
  const uint32_t off = uint32_t(((lane & 15) * a.r + rb) * 4);
  if (avec) {
    const f32x4 u = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, int(off), 0, 0));
    const f32x4 w = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, int(off + 16), 0, 0));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = u[e];
      x[4 + e] = w[e];
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) {  // unconditional loads, then ranks >= r are zeroed
      const float v = gld(r, off + 4 * e);
      x[e] = rb + e < a.r ? v : 0.f;
    }
  }
}

// B operand of one K-step and column block cb: B[32 ks + 8 (l / 16) + e][col of MFMA row l % 16]
// (zero past r or k).
__device__ __forceinline__ void load_b(float (&y)[8], const GridArgs& a, int64_t col0, int cb, int ks) {
  const int lane = threadIdx.x & 63, i = lane & 15;
  const int64_t lc = 16 * (i >> 2) + 4 * cb + (i & 3);
  const int rb = 32 * ks + 8 * (lane >> 4);
  const auto r = grid_rsrc(a.B + col0, int64_t(a.r) * a.k * 4 - col0 * 4);
  // unconditional loads (ranks >= r lie past the buffer's range and read as
  // zeros), then columns >= k are zeroed: no branch around a load
  const bool col_ok = col0 + lc < a.k;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float v = gld(r, uint32_t(((rb + e) * a.k + lc) * 4));
    y[e] = col_ok ? v : 0.f;
  }
}

// Bytes 0..3 of the result: bit 7 is the sign of x[0..3].
__device__ __forceinline__ uint32_t sign_bytes(const f32x4& x) {
  const uint32_t lo = __builtin_amdgcn_perm(__float_as_uint(x[1]), __float_as_uint(x[0]), 0x0c0c0703u);
  const uint32_t hi = __builtin_amdgcn_perm(__float_as_uint(x[3]), __float_as_uint(x[2]), 0x07030c0cu);
  return lo | hi;
}

// Two words of four nibble-bytes each -> one word of eight nibbles (element 0 lowest).
__device__ __forceinline__ uint32_t pack_nibble_bytes(uint32_t q0, uint32_t q1) {
  return __builtin_amdgcn_perm(q1 | (q1 >> 4), q0 | (q0 >> 4), 0x06040200u);
}

// Rounding decision, clip, packing and mask of one 16 x 64 wave tile, by the
// cheapest of the paths that is exact for the whole wave (INT-b Phi0 whose
// |delta| bound is below 1/2 on the whole tile has been copied already):
//  * delta identically zero on the strip (B = 0, the adapters' initial
//    state): round-half-even of Phi0, decided in integers;
//  * byte-parallel (swar_grid_q8): every |delta| is below the distance of the
//    non-tie codes to their rounding points and, at ties, above the error bound
//    tau, so only a tie depends on delta, through its sign; INT4 Phi0 is then q
//    itself.  Codes that would round off the grid send the wave on;
//  * per element: with Phi0 = n + cf 2^-f (n = floor, cf the f fraction bits),
//    u = n + 1/2 + w and w = (cf 2^-f - 1/2) + delta, one fused multiply-add of
//    exact terms; for w strictly between the integers j - 1 and j the nearest
//    integer to u is n + j = n + ceil(w).  That is certain unless w lies within
//    the error bound of an integer; a wave with such an element redoes its tile
//    with exact margins and float64 deltas (rare).
// The lane's results for its 16 columns: q as 16 nibbles (w0, w1) or 16 bytes
// (qb, Q8OUT), and the clip-mask bits.
struct GridOut {
  uint32_t w0, w1;
  uint32_t qb[4];
  uint32_t mb;
};

template <bool PACKED, bool MASK, bool B4, bool Q8OUT>
__device__ __forceinline__ void grid_decide(const GridArgs& a, const PhiRegs& P, const f32x4 (&acc)[4], float tau,
                                            bool zero_delta, int64_t row, int64_t c16, bool small_delta,
                                            GridOut& o) {
  const int bits = B4 ? 4 : a.bits;  // B4: the common 4-bit grid, constant for the compiler
  const int lo = -(1 << (bits - 1)), hi = (1 << (bits - 1)) - 1;
  const int f = PACKED ? 0 : 8 - bits;
  const bool row_ok = row < a.m;
  const int kin = int(max<int64_t>(0, min<int64_t>(16, a.k - c16)));  // the lane's columns inside k
  auto n_of = [&](int idx) { return PACKED ? phi_code<true>(P, idx) : phi_code<false>(P, idx) >> f; };

  int ut[16];
  uint32_t w0 = 0, w1 = 0;    // 16 nibbles (q as int4)
  uint32_t qb[4] = {0, 0, 0, 0};  // 16 bytes (q as int8, Q8OUT)
  uint32_t mb = 0;            // clip-mask bits of the lane's 16 columns
  bool done = false;  // q words (and an all-ones mask) already formed by the byte-parallel path
  if constexpr (PACKED) {
    if (small_delta) {  // the wave tile's |delta| is provably below 1/2: q is Phi0
      w0 = P.w[0];
      w1 = P.w[1];
      mb = 0xFFFFu;
      done = true;
    }
  }
  if (!done && !zero_delta) {
    // the regime of the byte-parallel path: every |delta| below the distance of the non-tie
    // codes to their rounding points and above the error bound (so its sign is certain)
    const float tz = fmaxf(tau, 0.f);
    float amx = 0.f, amn = __builtin_inff();
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        amx = fmaxf(amx, fabsf(acc[cb][v]));
        amn = fminf(amn, fabsf(acc[cb][v]));
      }
    const float ac = fabsf(a.c);
    const float lim = (PACKED ? 0.5f : __builtin_bit_cast(float, uint32_t(127 - f) << 23)) - tz - 0x1p-22f;
    // INT4 codes have no ties: inside the regime q does not depend on delta at all
    const bool fast = amx * ac < lim && (PACKED || amn * ac > tz) && a.c != 0.f && (!PACKED || bits == 4);
    bool regime = amx * ac < lim && a.c != 0.f && (!PACKED || bits == 4);
    if constexpr (!PACKED) {
      // A wave whose smallest |delta| is within the bound may still be decidable: only ties
      // (cf = 2^(f-1)) depend on delta, so check ties against the bound element by element.
      if (__builtin_amdgcn_ballot_w64(!fast) && !__builtin_amdgcn_ballot_w64(!regime)) {
        const uint32_t ones = 0x01010101u;
        // covers the rounding of c * acc; never 0, so that a tie with delta exactly 0 is caught
        const float tzu = fmaxf(tz * (1.f + 0x1p-20f), 0x1p-100f);
        uint32_t bad = 0;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          f32x4 d;
#pragma unroll
          for (int v = 0; v < 4; ++v) d[v] = __builtin_fmaf(fabsf(acc[g][v]), ac, -tzu);  // < 0: within the bound
          const uint32_t y = (P.w[g] & (ones * ((1u << f) - 1))) ^ (ones << (f - 1));  // 0 in tie bytes
          const uint32_t tie = ~((y + 0x7F7F7F7Fu) | y) & 0x80808080u;
          bad |= sign_bytes(d) & tie;
        }
        regime = bad == 0;
      } else {
        regime = fast;
      }
    }
    if (!__builtin_amdgcn_ballot_w64(!(PACKED ? fast : regime))) {
      if constexpr (PACKED) {
        // |delta| < 1/2: q is Phi0 itself (INT4 codes are always on the grid)
        w0 = P.w[0];
        w1 = P.w[1];
        done = true;
      } else {
        uint32_t q[4], clip = 0;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const uint32_t sb = sign_bytes(acc[g]);
          const uint32_t incb = ((a.c > 0.f ? ~sb : sb) >> 7) & 0x01010101u;
          q[g] = swar_grid_q8(P.w[g], incb, f, bits, clip);
        }
        if (!__builtin_amdgcn_ballot_w64(clip != 0)) {
          if constexpr (Q8OUT) {
#pragma unroll
            for (int g = 0; g < 4; ++g) qb[g] = q[g];
          } else {
            w0 = pack_nibble_bytes(q[0], q[1]);
            w1 = pack_nibble_bytes(q[2], q[3]);
          }
          done = true;
        }
      }
      if (done) mb = 0xFFFFu;  // inside the regime every rounded value is on the grid
    }
  }
  if (done) {
  } else if (zero_delta) {
    // round-half-even of Phi0 = n + cf 2^-f
    const int half = f ? 1 << (f - 1) : 0;
#pragma unroll
    for (int idx = 0; idx < 16; ++idx) {
      const int code = phi_code<PACKED>(P, idx), n = code >> f, cf = code & ((1 << f) - 1);
      ut[idx] = f ? n + int(cf > half || (cf == half && (n & 1))) : code;
    }
  } else {
    const float tz = fmaxf(tau, 0.f);
    const float sf = __builtin_bit_cast(float, uint32_t(127 - f) << 23);  // 2^-f
    uint64_t flag = 0;
    // fraction bits of the four codes of each word, as unsigned bytes (Q8 only)
    uint32_t fw[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) fw[q] = P.w[q] & (0x01010101u * uint32_t((1 << f) - 1));
#pragma unroll
    for (int idx = 0; idx < 16; ++idx) {
      const float x = PACKED ? -0.5f : __builtin_fmaf(float((fw[idx >> 2] >> (8 * (idx & 3))) & 0xffu), sf, -0.5f);
      // u = n + 1/2 + w: for w in (j - 1, j), j an integer, the nearest integer to u is n + j =
      // n + ceil(w); certain unless w lies within the bound of an integer (the bound adds the
      // rounding of this fused multiply-add, below 2^-24 |w|, doubled)
      const float w = __builtin_fmaf(acc[idx >> 2][idx & 3], a.c, x);
      flag |= __builtin_amdgcn_ballot_w64(fabsf(w - __builtin_rintf(w)) <= __builtin_fmaf(0x1p-23f, fabsf(w), tz));
      ut[idx] = n_of(idx) + int(__builtin_ceilf(w));
    }
    if (flag) {
      // exact margins and float64 re-decision for the lanes' elements within the bound
      uint32_t need = 0;
#pragma unroll
      for (int idx = 0; idx < 16; ++idx) {
        float margin;
        ut[idx] = grid_round(phi_code<PACKED>(P, idx), f, a.c * acc[idx >> 2][idx & 3], &margin);
        need |= uint32_t(margin <= tau && row_ok && idx < kin) << idx;
      }
      while (__builtin_amdgcn_ballot_w64(need != 0)) {
        const bool mine = need != 0;
        const int idx = mine ? __builtin_ctz(need) : -1;
        need &= need - 1;
        int unew = 0;
        if (mine) {
          const int64_t col = c16 + idx;
          const float* Ar = a.A + row * a.r;
          const float* Bc = a.B + col;
          double d0 = 0.0, d1 = 0.0, d2 = 0.0, d3 = 0.0;  // independent partial sums keep the loads in flight
          int rho = 0;
#pragma unroll 1
          for (; rho + 4 <= a.r; rho += 4) {
            d0 = __builtin_fma(double(Ar[rho]), double(Bc[int64_t(rho) * a.k]), d0);
            d1 = __builtin_fma(double(Ar[rho + 1]), double(Bc[int64_t(rho + 1) * a.k]), d1);
            d2 = __builtin_fma(double(Ar[rho + 2]), double(Bc[int64_t(rho + 2) * a.k]), d2);
            d3 = __builtin_fma(double(Ar[rho + 3]), double(Bc[int64_t(rho + 3) * a.k]), d3);
          }
#pragma unroll 1
          for (; rho < a.r; ++rho) d0 = __builtin_fma(double(Ar[rho]), double(Bc[int64_t(rho) * a.k]), d0);
          unew = grid_round_f64(phi_code_dyn<PACKED>(P, idx), f, a.c64 * ((d0 + d1) + (d2 + d3)));
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) ut[j] = j == idx ? unew : ut[j];
      }
    }
  }

  // Clip and pack 16 nibbles (8 bytes) or 16 bytes (Q8OUT); columns >= k are
  // written as 0.  Mask: bit idx of the lane's 16-bit word is [the rounded value
  // of column c16 + idx lies on the grid].
  if (!done) {
#pragma unroll
    for (int idx = 0; idx < 16; ++idx) {
      const int q = min(max(ut[idx], lo), hi);
      if constexpr (Q8OUT) {
        qb[idx >> 2] |= uint32_t(q & 255) << (8 * (idx & 3));
      } else {
        const uint32_t nib = uint32_t(q & 15) << (4 * (idx & 7));
        if (idx < 8) w0 |= nib;
        else w1 |= nib;
      }
      if constexpr (MASK) mb |= uint32_t(q == ut[idx]) << idx;
    }
  }
  if (kin < 16) {
    if constexpr (Q8OUT) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int nb = kin - 4 * g;  // bytes of word g inside k
        qb[g] &= nb >= 4 ? 0xFFFFFFFFu : nb <= 0 ? 0u : (1u << (8 * nb)) - 1u;
      }
    } else {
      const uint64_t keep = (uint64_t(1) << (4 * kin)) - 1;  // kin <= 15
      w0 &= uint32_t(keep);
      w1 &= uint32_t(keep >> 32);
    }
  }
  o.w0 = w0;
  o.w1 = w1;
#pragma unroll
  for (int g = 0; g < 4; ++g) o.qb[g] = qb[g];
  o.mb = mb;
}

// Stores one lane's 16 columns of q (and mask) at row, columns c16 .. c16 + 15.
template <bool MASK, bool Q8OUT>
__device__ __forceinline__ void grid_store(const GridArgs& a, const GridOut& o, int64_t row, int64_t c16) {
  const uint32_t w0 = o.w0, w1 = o.w1, mb = o.mb;
  uint32_t qb[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) qb[g] = o.qb[g];
  if (row < a.m && c16 < a.kq) {
    if constexpr (Q8OUT) {
      uint8_t* dst = a.qout + row * a.ldq + c16;
      if (c16 + 16 <= a.kq && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
        *reinterpret_cast<u32x4*>(dst) = u32x4{qb[0], qb[1], qb[2], qb[3]};
      } else {
        const int64_t nbytes = min<int64_t>(16, a.kq - c16);
        for (int64_t b = 0; b < nbytes; ++b) dst[b] = uint8_t(qb[b >> 2] >> (8 * (b & 3)));
      }
    } else {
      uint8_t* dst = a.qout + row * a.ldq + (c16 >> 1);
      if (c16 + 16 <= a.kq && (reinterpret_cast<uintptr_t>(dst) & 7) == 0) {
        *reinterpret_cast<u32x2*>(dst) = u32x2{w0, w1};
      } else {
        const int64_t nbytes = min<int64_t>(8, (a.kq - c16 + 1) >> 1);
        for (int64_t b = 0; b < nbytes; ++b) dst[b] = uint8_t((b < 4 ? w0 : w1) >> (8 * (b & 3)));
      }
    }
    if constexpr (MASK) a.mout[row * a.ldm + (c16 >> 4)] = uint16_t(mb);
  }
}

template <bool PACKED, bool MASK, bool B4, bool Q8OUT>
__device__ __forceinline__ void grid_finish(const GridArgs& a, const PhiRegs& P, const f32x4 (&acc)[4], float tau,
                                            bool zero_delta, int64_t row, int64_t c16, bool small_delta = false) {
  GridOut o;
  grid_decide<PACKED, MASK, B4, Q8OUT>(a, P, acc, tau, zero_delta, row, c16, small_delta, o);
  grid_store<MASK, Q8OUT>(a, o, row, c16);
}

// COAL (r = 32, 16-byte aligned A and B rows, k % 4 == 0): B and A are read
// with coalesced 16-byte loads and rearranged into MFMA operand order in the
// wave's LDS region; otherwise each lane loads its own operand values.
template <bool PACKED, bool ONEK, bool MASK, bool COAL, bool B4, bool Q8OUT>
__global__ __launch_bounds__(GR_THREADS) void k_grid(GridArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  // the block's 4 waves cover 256 adjacent columns (whole 128-byte lines of q
  // and of Q8 Phi0) of the same nit 16-row blocks
  const int64_t nstrips = (a.kq + 4 * GR_COLS - 1) / (4 * GR_COLS);
  const int64_t col0 = int64_t(blockIdx.x % nstrips) * 4 * GR_COLS + GR_COLS * wave;
  const int64_t rb0 = int64_t(blockIdx.x / nstrips) * a.nit;  // first 16-row block of the block
  const int64_t c16 = col0 + 16 * (lane >> 4);                // the lane's first column
  const int nks = (a.r + 31) / 32;
  const bool avec = (a.r & 31) == 0 && (reinterpret_cast<uintptr_t>(a.A) & 15) == 0;
  // 16-byte (8-byte) code loads need aligned rows; loads past the end of a row
  // only feed columns >= k, which are never used
  const bool pvec = ((a.ld_phi | int64_t(reinterpret_cast<uintptr_t>(a.phi0))) & (PACKED ? 7 : 15)) == 0;

  // The wave's B columns: for r <= 32 (one K-step) their bf16 hi/lo fragments
  // stay in the wave's own LDS region for all its rounds, else they are
  // reloaded per K-step.  The largest column norm and |B| of the wave's 64
  // columns bound the error.
  __shared__ __attribute__((aligned(16))) u32x4 bfrag[4][2][4][64];
  __shared__ __attribute__((aligned(16))) float arow[COAL ? 4 : 1][16][36];  // COAL: the tile's A rows (144-byte pitch)
  float bss = 0.f, bmx = 0.f;
  if constexpr (COAL) {
    // B[0..31][col0 .. col0 + 63]: 8 loads of 4 rank rows x 256 bytes, staged raw
    // in the wave's fragment region, then read back in operand order
    float* raw = reinterpret_cast<float*>(&bfrag[wave][0][0][0]);
    const auto rb = grid_rsrc(a.B + col0, int64_t(a.r) * a.k * 4 - col0 * 4);
    const int cl = 4 * (lane & 15);
    u32x4 v[8];
#pragma unroll
    for (int t = 0; t < 8; ++t)
      v[t] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                           rb, int(uint32_t(((4 * t + (lane >> 4)) * a.k + cl) * 4)), 0, 0));
#pragma unroll
    for (int t = 0; t < 8; ++t) {
#pragma unroll
      for (int j = 0; j < 4; ++j) v[t][j] = col0 + cl + j < a.k ? v[t][j] : 0u;
      *reinterpret_cast<u32x4*>(raw + (4 * t + (lane >> 4)) * 64 + cl) = v[t];
    }
    float y[4][8];
    float ss[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        y[cb][e] = raw[(8 * (lane >> 4) + e) * 64 + 16 * ((lane & 15) >> 2) + 4 * cb + (lane & 3)];
        ss[cb] = __builtin_fmaf(y[cb][e], y[cb][e], ss[cb]);
        bmx = fmaxf(bmx, fabsf(y[cb][e]));
      }
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      u32x4 h, l;
      split8(y[cb], h, l);
      bfrag[wave][0][cb][lane] = h;
      bfrag[wave][1][cb][lane] = l;
      ss[cb] += __shfl_xor(ss[cb], 16);
      ss[cb] += __shfl_xor(ss[cb], 32);
      bss = fmaxf(bss, ss[cb]);
    }
    for (int off = 1; off < 64; off <<= 1) {
      bss = fmaxf(bss, __shfl_xor(bss, off));
      bmx = fmaxf(bmx, __shfl_xor(bmx, off));
    }
  } else {
    float ss[4] = {0.f, 0.f, 0.f, 0.f};
    for (int ks = 0; ks < nks; ++ks) {
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        float y[8];
        load_b(y, a, col0, cb, ks);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          ss[cb] = __builtin_fmaf(y[e], y[e], ss[cb]);
          bmx = fmaxf(bmx, fabsf(y[e]));
        }
        if (ONEK) {
          u32x4 h, l;
          split8(y, h, l);
          bfrag[wave][0][cb][lane] = h;
          bfrag[wave][1][cb][lane] = l;
        }
      }
    }
    // the 4 lanes l % 16 + 16 g hold the 4 rank slices of a column
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      ss[cb] += __shfl_xor(ss[cb], 16);
      ss[cb] += __shfl_xor(ss[cb], 32);
      bss = fmaxf(bss, ss[cb]);
    }
    for (int off = 1; off < 64; off <<= 1) {
      bss = fmaxf(bss, __shfl_xor(bss, off));
      bmx = fmaxf(bmx, __shfl_xor(bmx, off));
    }
  }
  const float nb = norm_bound(bss, bmx, a.r);

  int64_t rowblk = rb0;
  PhiRegs P;
  float xa[8];
  u32x4 xc[2];  // COAL: the 16 A rows of a tile, rows lane / 8 and 8 + lane / 8, 16-byte chunk lane % 8
  auto load_a_coal = [&](int64_t rblk) {
    const auto r = grid_rsrc(a.A + rblk * 16 * 32, (a.m - rblk * 16) * 128);
#pragma unroll
    for (int h = 0; h < 2; ++h)
      xc[h] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, 1024 * h + 16 * lane, 0, 0));
  };
  load_phi<PACKED>(P, a, rowblk, col0, pvec);
  if constexpr (COAL) load_a_coal(rowblk);
  else if (ONEK) load_a(xa, a, rowblk, 0, avec);
  for (int it = 0; it < a.nit; ++it, ++rowblk) {
    if (rowblk * 16 >= a.m) break;  // wave-uniform
    const int64_t row = rowblk * 16 + (lane & 15);
    f32x4 acc[4];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    float ass = 0.f, amx = 0.f;
    const PhiRegs Pc = P;
    if (ONEK) {
      float x[8];
      if constexpr (COAL) {
        // through the wave's LDS rows: lane l takes row l % 16, ranks 8 (l / 16) .. +7
#pragma unroll
        for (int h = 0; h < 2; ++h) *reinterpret_cast<u32x4*>(&arow[wave][8 * h + (lane >> 3)][4 * (lane & 7)]) = xc[h];
        const f32x4 u = *reinterpret_cast<const f32x4*>(&arow[wave][lane & 15][8 * (lane >> 4)]);
        const f32x4 w = *reinterpret_cast<const f32x4*>(&arow[wave][lane & 15][8 * (lane >> 4) + 4]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[e] = u[e];
          x[4 + e] = w[e];
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = xa[e];
      }
      // prefetch the next round's Phi0 codes and A slice
      if (it + 1 < a.nit) {
        load_phi<PACKED>(P, a, rowblk + 1, col0, pvec);
        if constexpr (COAL) load_a_coal(rowblk + 1);
        else load_a(xa, a, rowblk + 1, 0, avec);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        ass = __builtin_fmaf(x[e], x[e], ass);
        amx = fmaxf(amx, fabsf(x[e]));
      }
      // row norm: the 4 lanes l % 16 + 16 g hold the 4 rank slices of the row
      ass += __shfl_xor(ass, 16);
      ass += __shfl_xor(ass, 32);
      amx = fmaxf(amx, __shfl_xor(amx, 16));
      amx = fmaxf(amx, __shfl_xor(amx, 32));
      bool small = false;
      if constexpr (PACKED) {
        // integer Phi0: |delta| <= |c| ||A_i|| ||B_j|| below 1/2 on the whole wave tile means
        // q = Phi0 (no rounding can move, nothing clips), decided without the product
        const float bound = fabsf(a.c) * norm_bound(ass, amx, a.r) * nb * 1.02f;
        // (4-bit grids only: a narrower grid may clip an INT4 code of Phi0)
        small = (B4 || a.bits == 4) && !__builtin_amdgcn_ballot_w64(!(bound < 0.5f - 0x1p-20f));
      }
      if (small) {
        grid_finish<PACKED, MASK, B4, Q8OUT>(a, Pc, acc, 0.f, false, row, c16, true);
        continue;
      }
      u32x4 ah, al;
      split8(x, ah, al);
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        const u32x4 ph = bfrag[wave][0][cb][lane], pl = bfrag[wave][1][cb][lane];
        acc[cb] = mfma16(ph, ah, acc[cb]);
        acc[cb] = mfma16(pl, ah, acc[cb]);
        acc[cb] = mfma16(ph, al, acc[cb]);
      }
    } else {
      if (it + 1 < a.nit) load_phi<PACKED>(P, a, rowblk + 1, col0, pvec);
      for (int ks = 0; ks < nks; ++ks) {
        float x[8];
        load_a(x, a, rowblk, ks, avec);
        u32x4 ah, al;
        split8(x, ah, al);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          ass = __builtin_fmaf(x[e], x[e], ass);
          amx = fmaxf(amx, fabsf(x[e]));
        }
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
          float y[8];
          load_b(y, a, col0, cb, ks);
          u32x4 ph, pl;
          split8(y, ph, pl);
          acc[cb] = mfma16(ph, ah, acc[cb]);
          acc[cb] = mfma16(pl, ah, acc[cb]);
          acc[cb] = mfma16(ph, al, acc[cb]);
        }
      }
      // row norm: the 4 lanes l % 16 + 16 g hold the 4 rank slices of the row
      ass += __shfl_xor(ass, 16);
      ass += __shfl_xor(ass, 32);
      amx = fmaxf(amx, __shfl_xor(amx, 16));
      amx = fmaxf(amx, __shfl_xor(amx, 32));
    }
    // -1 where delta is exactly zero (a zero A row or zero B columns, e.g. B at its zero
    // initialisation), so that no element is re-decided there
    const float tau = amx == 0.f ? -1.f : a.tau_coef * norm_bound(ass, amx, a.r) * nb;
    grid_finish<PACKED, MASK, B4, Q8OUT>(a, Pc, acc, tau, bmx == 0.f, row, c16);
  }
}

// Wide tiles, for r = 32 with 16-byte aligned A and B rows, k % 4 == 0 and
// 16-byte aligned Phi0 rows.
// A block owns 256 adjacent columns (a strip) and 4 nit consecutive 16-row
// blocks; wave w takes row blocks 4 it + w across the whole strip, so that one
// 16-row A slice serves 4096 outputs.  The strip is computed as four
// sub-tiles of 16 x 64 (sixteen 16x16 MFMA tiles) whose B columns are
// assigned so that lane l owns 64 consecutive columns, 64 (l / 16) .. +63,
// of weight row l % 16: in sub-tile j, MFMA row i of column block cb stands
// for strip column 64 (i / 4) + 16 j + 4 cb + i % 4.  A lane's Phi0 codes,
// q nibbles and mask words of the strip are then 32 (64) contiguous bytes,
// moved with 16-byte accesses that cover whole 128-byte lines per row.  Wave w
// builds the B fragments of sub-tile w in LDS; all four waves read all four.
// Blocks are numbered so that each XCD (blocks are dispatched round-robin
// over the 8 XCDs) takes a contiguous range of row blocks, keeping the A rows
// in one L2.  The decision per sub-tile is grid_decide, as in k_grid.
template <bool PACKED>
__device__ __forceinline__ void load_phi_w(PhiRegs (&P)[4], const GridArgs& a, int64_t rowblk, int64_t strip0) {
  const int lane = threadIdx.x & 63, g = lane >> 4;
  const int64_t row0 = rowblk * 16, cb0 = PACKED ? strip0 / 2 : strip0;
  const auto r = grid_rsrc(a.phi0 + row0 * a.ld_phi + cb0, (a.m - row0) * a.ld_phi - cb0);
  // the lane's bytes: 32 g .. +31 (packed) or 64 g .. +63 (Q8) of the row's strip
  const uint32_t off = uint32_t((lane & 15) * a.ld_phi + (PACKED ? 32 : 64) * g);
#pragma unroll
  for (int h = 0; h < (PACKED ? 2 : 4); ++h) {
    const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, int(off + 16 * h), 0, 0));
    if constexpr (PACKED) {
      P[2 * h] = PhiRegs{{v[0], v[1], 0u, 0u}};
      P[2 * h + 1] = PhiRegs{{v[2], v[3], 0u, 0u}};
    } else {
      P[h] = PhiRegs{{v[0], v[1], v[2], v[3]}};
    }
  }
}

template <bool PACKED, bool MASK, bool B4, bool Q8OUT, bool MULTI>
__global__ __launch_bounds__(GR_THREADS) void k_grid_w(GridArgs a) {
  const int lane = threadIdx.x & 63, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  // logical block: XCD x = blockIdx % 8 takes the contiguous range starting at x floor(N/8) + min(x, N % 8)
  const int64_t nblk = gridDim.x, x = blockIdx.x % 8;
  const int64_t lb = x * (nblk / 8) + min<int64_t>(x, nblk % 8) + blockIdx.x / 8;
  const int64_t nstrips = (a.kq + 4 * GR_COLS - 1) / (4 * GR_COLS);
  const int64_t strip0 = (lb % nstrips) * 4 * GR_COLS;
  const int64_t rb0 = (lb / nstrips) * 4 * a.nit + wave;  // the wave's first 16-row block
  const int nks = MULTI ? a.r / 32 : 1;                       // 32-rank chunks (MULTI: r a multiple of 32)

  __shared__ __attribute__((aligned(16))) u32x4 bfrag[4][2][4][64];
  __shared__ __attribute__((aligned(16))) float arow[4][16][36];  // the wave's A rows (144-byte pitch)
  __shared__ float nbs[4];                                         // column-norm bound per sub-tile
  __shared__ float cnb[4], cna[4];                                 // block-wide copy test: B and A norm bounds per wave

  // round 0's codes and A rows first: they do not depend on the B fragments
  PhiRegs P[4];
  u32x4 xc[2];  // 16 A rows x 32 ranks of a round: rows lane / 8 and 8 + lane / 8, 16-byte chunk lane % 8
  auto load_a_chunk = [&](int64_t rblk, int ch) {
    const auto r = grid_rsrc(a.A + rblk * 16 * a.r, (a.m - rblk * 16) * int64_t(a.r) * 4);
#pragma unroll
    for (int h = 0; h < 2; ++h)
      xc[h] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                            r, int(uint32_t((8 * h + (lane >> 3)) * a.r * 4 + 128 * ch + 16 * (lane & 7))),
                                            0, 0));
  };
  auto load_round = [&](int64_t rblk) {
    load_phi_w<PACKED>(P, a, rblk, strip0);
    load_a_chunk(rblk, 0);
  };
  load_round(rb0);

  // B[32 ch .. 32 ch + 31] at the strip columns 64 q + 16 w + c (q = 0..3, c = 0..15) of
  // sub-tile w: 8 loads of 4 rank rows, staged raw (rank row-major, 64 floats, position
  // 16 q + c) in the wave's fragment region, then read back in operand order.  ssc[cb]
  // accumulates the squared norm of the lane's column of block cb, bmx the largest |B|.
  float ssc[4] = {0.f, 0.f, 0.f, 0.f}, bmx = 0.f;
  auto load_b = [&](int ch, u32x4 (&v)[8]) {
    const auto rb = grid_rsrc(a.B + strip0, int64_t(a.r) * a.k * 4 - strip0 * 4);
    const int64_t gc = 64 * ((lane & 15) >> 2) + 16 * wave + 4 * (lane & 3);  // strip column
#pragma unroll
    for (int t = 0; t < 8; ++t)
      v[t] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                           rb, int(uint32_t(((32 * ch + 4 * t + (lane >> 4)) * a.k + gc) * 4)), 0, 0));
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j) v[t][j] = strip0 + gc + j < a.k ? v[t][j] : 0u;
  };
  auto stage_b_tail = [&]() {
    const float* raw = reinterpret_cast<const float*>(&bfrag[wave][0][0][0]);
    float y[4][8];
    float ss[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        y[cb][e] = raw[(8 * (lane >> 4) + e) * 64 + 16 * ((lane & 15) >> 2) + 4 * cb + (lane & 3)];
        ss[cb] = __builtin_fmaf(y[cb][e], y[cb][e], ss[cb]);
        bmx = fmaxf(bmx, fabsf(y[cb][e]));
      }
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      u32x4 h, l;
      split8(y[cb], h, l);
      bfrag[wave][0][cb][lane] = h;
      bfrag[wave][1][cb][lane] = l;
      ss[cb] += __shfl_xor(ss[cb], 16);
      ss[cb] += __shfl_xor(ss[cb], 32);
      ssc[cb] += ss[cb];
    }
  };
  auto stage_b_from = [&](const u32x4 (&v)[8]) {
    float* raw = reinterpret_cast<float*>(&bfrag[wave][0][0][0]);
    const int cl = 4 * (lane & 15);  // raw position
#pragma unroll
    for (int t = 0; t < 8; ++t) *reinterpret_cast<u32x4*>(raw + (4 * t + (lane >> 4)) * 64 + cl) = v[t];
    stage_b_tail();
  };
  // load_b + stage_b_from in one, with each raw write next to its load (the byte-parallel and
  // multi-chunk paths keep this form: split, they need more registers)
  auto stage_b = [&](int ch) {
    float* raw = reinterpret_cast<float*>(&bfrag[wave][0][0][0]);
    const auto rb = grid_rsrc(a.B + strip0, int64_t(a.r) * a.k * 4 - strip0 * 4);
    const int cl = 4 * (lane & 15);                                             // raw position
    const int64_t gc = 64 * ((lane & 15) >> 2) + 16 * wave + 4 * (lane & 3);  // strip column
    u32x4 v[8];
#pragma unroll
    for (int t = 0; t < 8; ++t)
      v[t] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                           rb, int(uint32_t(((32 * ch + 4 * t + (lane >> 4)) * a.k + gc) * 4)), 0, 0));
#pragma unroll
    for (int t = 0; t < 8; ++t) {
#pragma unroll
      for (int j = 0; j < 4; ++j) v[t][j] = strip0 + gc + j < a.k ? v[t][j] : 0u;
      *reinterpret_cast<u32x4*>(raw + (4 * t + (lane >> 4)) * 64 + cl) = v[t];
    }
    stage_b_tail();
  };
  // the sub-tile's column-norm bound from the accumulated column sums (0 exactly when its B
  // columns are all zero), shared through LDS
  auto publish_nb = [&]() {
    float bss = fmaxf(fmaxf(ssc[0], ssc[1]), fmaxf(ssc[2], ssc[3])), m = bmx;
    for (int off = 1; off < 64; off <<= 1) {
      bss = fmaxf(bss, __shfl_xor(bss, off));
      m = fmaxf(m, __shfl_xor(m, off));
    }
    if (lane == 0) nbs[wave] = norm_bound(bss, m, a.r);
  };
  // the lane's 8 ranks of its row (row l % 16, ranks 8 (l / 16) .. +7 of the chunk), through
  // the wave's LDS rows
  auto a_slice = [&](float (&xv)[8]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) *reinterpret_cast<u32x4*>(&arow[wave][8 * h + (lane >> 3)][4 * (lane & 7)]) = xc[h];
    const f32x4 u = *reinterpret_cast<const f32x4*>(&arow[wave][lane & 15][8 * (lane >> 4)]);
    const f32x4 w = *reinterpret_cast<const f32x4*>(&arow[wave][lane & 15][8 * (lane >> 4) + 4]);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      xv[e] = u[e];
      xv[4 + e] = w[e];
    }
  };

  // q [row][cl0 .. cl0 + 63] (and the mask words) of one round, as the round loop below stores
  // them (which keeps its own copy of these stores: through this lambda it needs more registers)
  auto store_round = [&](int64_t row, int64_t cl0, const GridOut (&out)[4]) {
    const bool whole = row < a.m && cl0 + 64 <= a.kq;
    if constexpr (Q8OUT) {
      uint8_t* dst = a.qout + row * a.ldq + cl0;
      if (whole && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<u32x4*>(dst + 16 * j) = u32x4{out[j].qb[0], out[j].qb[1], out[j].qb[2], out[j].qb[3]};
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) grid_store<false, true>(a, out[j], row, cl0 + 16 * j);
      }
    } else {
      uint8_t* dst = a.qout + row * a.ldq + (cl0 >> 1);
      if (whole && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
          *reinterpret_cast<u32x4*>(dst + 16 * h) =
              u32x4{out[2 * h].w0, out[2 * h].w1, out[2 * h + 1].w0, out[2 * h + 1].w1};
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) grid_store<false, false>(a, out[j], row, cl0 + 16 * j);
      }
    }
    if constexpr (MASK) {
      uint16_t* md = a.mout + row * a.ldm + (cl0 >> 4);
      if (whole && (reinterpret_cast<uintptr_t>(md) & 7) == 0) {
        *reinterpret_cast<u32x2*>(md) =
            u32x2{(out[0].mb & 0xFFFFu) | (out[1].mb << 16), (out[2].mb & 0xFFFFu) | (out[3].mb << 16)};
      } else if (row < a.m) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (cl0 + 16 * j < a.kq) md[j] = uint16_t(out[j].mb);
      }
    }
  };

  float nbv[4];
  f32x4 acc4[4][4];  // MULTI: the products of all rank chunks, per sub-tile
  float ass = 0.f, amx = 0.f;
  u32x4 ah, al;
  if constexpr (!MULTI) {
    u32x4 bv[8];
    if constexpr (PACKED) load_b(0, bv);
    else stage_b(0);
    if constexpr (PACKED) {
      // Integer Phi0 on a 4-bit grid: when |c| max_i ||A_i|| max_j ||B_j|| over all rows of the
      // block's rounds and all columns of its strip is below 1/2, every sub-tile has q = Phi0 and
      // nothing clips (the per-sub-tile test below would pass everywhere), so the block copies
      // Phi0 without staging B fragments.  The test uses maxima of the same norm bounds and covers
      // up to four rounds (the launcher's largest nit).
      if ((B4 || a.bits == 4) && a.nit <= 4) {
        // column sums of squares of the wave's sub-tile, straight from the loaded values: lanes
        // l, l ^ 16, l ^ 32, l ^ 48 hold the 32 ranks of the same 4 columns
        float cs[4] = {0.f, 0.f, 0.f, 0.f}, m = 0.f;
#pragma unroll
        for (int t = 0; t < 8; ++t)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float x = __uint_as_float(bv[t][j]);
            cs[j] = __builtin_fmaf(x, x, cs[j]);
            m = fmaxf(m, fabsf(x));
          }
        float bss = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          cs[j] += __shfl_xor(cs[j], 16);
          cs[j] += __shfl_xor(cs[j], 32);
          bss = fmaxf(bss, cs[j]);
        }
        // largest row sum of squares of 16 A rows held as the round's chunks (lanes 8 e .. 8 e + 7
        // hold the eight 16-byte chunks of rows e and 8 + e)
        float ras = 0.f, ram = 0.f;
        auto rows_max = [&](const u32x4 (&v)[2]) {
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            float ss = 0.f, mx = 0.f;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float x = __uint_as_float(v[h][e]);
              ss = __builtin_fmaf(x, x, ss);
              mx = fmaxf(mx, fabsf(x));
            }
#pragma unroll
            for (int off = 1; off < 8; off <<= 1) {
              ss += __shfl_xor(ss, off);
              mx = fmaxf(mx, __shfl_xor(mx, off));
            }
            ras = fmaxf(ras, ss);
            ram = fmaxf(ram, mx);
          }
        };
        auto wave_max = [&](float& x) {
          for (int off = 1; off < 64; off <<= 1) x = fmaxf(x, __shfl_xor(x, off));
        };
        // first with round 0's rows (their A chunk is loaded): a block whose B columns and first
        // rows already exceed the bound goes on without loading the other rounds' rows
        rows_max(xc);
        wave_max(bss);
        wave_max(m);
        wave_max(ras);
        wave_max(ram);
        if (lane == 0) {
          cnb[wave] = norm_bound(bss, m, a.r);
          cna[wave] = norm_bound(ras, ram, a.r);
        }
        __syncthreads();
        const float nbm = fmaxf(fmaxf(cnb[0], cnb[1]), fmaxf(cnb[2], cnb[3]));
        const float lim = 0.5f - 0x1p-20f;
        if (fabsf(a.c) * fmaxf(fmaxf(cna[0], cna[1]), fmaxf(cna[2], cna[3])) * nbm * 1.02f < lim) {  // block-uniform
          // the other rounds' rows, and every round's codes, in flight at once (rows past m read 0)
          PhiRegs Pr[4][4];
#pragma unroll
          for (int j = 0; j < 4; ++j) Pr[0][j] = P[j];
          u32x4 av[4][2];
#pragma unroll
          for (int it = 1; it < 4; ++it) {
            const int64_t rblk = rb0 + 4 * it;
            const auto r = grid_rsrc(a.A + rblk * 16 * a.r, it < a.nit ? (a.m - rblk * 16) * int64_t(a.r) * 4 : 0);
#pragma unroll
            for (int h = 0; h < 2; ++h)
              av[it][h] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                        r, int(uint32_t((8 * h + (lane >> 3)) * a.r * 4 + 16 * (lane & 7))), 0, 0));
            if (it < a.nit) load_phi_w<PACKED>(Pr[it], a, rblk, strip0);
          }
#pragma unroll
          for (int it = 1; it < 4; ++it) rows_max(av[it]);
          wave_max(ras);
          wave_max(ram);
          __syncthreads();  // every wave has read the first round's values
          if (lane == 0) cna[wave] = norm_bound(ras, ram, a.r);
          __syncthreads();
          const float nam = fmaxf(fmaxf(cna[0], cna[1]), fmaxf(cna[2], cna[3]));
          if (fabsf(a.c) * nam * nbm * 1.02f < lim) {  // block-uniform
            const f32x4 zero[4] = {};
#pragma unroll
            for (int it = 0; it < 4; ++it) {
              const int64_t rowblk = rb0 + 4 * it;
              if (it >= a.nit || rowblk * 16 >= a.m) break;  // wave-uniform
              const int64_t row = rowblk * 16 + (lane & 15);
              GridOut out[4];
#pragma unroll
              for (int j = 0; j < 4; ++j)
                grid_decide<PACKED, MASK, B4, Q8OUT>(a, Pr[it][j], zero, 0.f, false, row, strip0 + 64 * g + 16 * j, true, out[j]);
              store_round(row, strip0 + 64 * g, out);
            }
            return;
          }
        }
      }
    }
    if constexpr (PACKED) stage_b_from(bv);
    publish_nb();
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) nbv[j] = nbs[j];
  } else {
    // one round per block (nit = 1); every wave takes part in every barrier, also a wave whose
    // rows lie past m (its loads read zeros and its stores are skipped)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) acc4[j][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int ch = 0; ch < nks; ++ch) {
      if (ch > 0) {
        __syncthreads();  // every wave is done with the previous chunk's fragments
        load_a_chunk(rb0, ch);
      }
      stage_b(ch);
      __syncthreads();
      float xv[8];
      a_slice(xv);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        ass = __builtin_fmaf(xv[e], xv[e], ass);
        amx = fmaxf(amx, fabsf(xv[e]));
      }
      split8(xv, ah, al);
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
          const u32x4 ph = bfrag[j][0][cb][lane], pl = bfrag[j][1][cb][lane];
          acc4[j][cb] = mfma16(ph, ah, acc4[j][cb]);
          acc4[j][cb] = mfma16(pl, ah, acc4[j][cb]);
          acc4[j][cb] = mfma16(ph, al, acc4[j][cb]);
        }
    }
    publish_nb();
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) nbv[j] = nbs[j];
  }
  const int64_t cl0_ = strip0 + 64 * g;  // the lane's first column

  int64_t rowblk = rb0;
  for (int it = 0; it < a.nit; ++it, rowblk += 4) {
    if (!MULTI && rowblk * 16 >= a.m) break;  // wave-uniform
    const int64_t row = rowblk * 16 + (lane & 15);
    // opaque per round, like the sub-tile index below: bounds and addresses derived
    // from the lane's columns are formed where they are used, not kept across rounds
    int64_t cl0 = cl0_;
    asm volatile("" : "+v"(cl0));
    PhiRegs Pc[4];
    if constexpr (!MULTI) {
      float xv[8];
      a_slice(xv);
#pragma unroll
      for (int j = 0; j < 4; ++j) Pc[j] = P[j];
      if (it + 1 < a.nit) load_round(rowblk + 4);
      ass = 0.f;
      amx = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        ass = __builtin_fmaf(xv[e], xv[e], ass);
        amx = fmaxf(amx, fabsf(xv[e]));
      }
      split8(xv, ah, al);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) Pc[j] = P[j];
    }
    // row norm: the 4 lanes l % 16 + 16 g hold the 4 rank slices of the row
    float rss = ass + __shfl_xor(ass, 16);
    rss += __shfl_xor(rss, 32);
    float rmx = fmaxf(amx, __shfl_xor(amx, 16));
    rmx = fmaxf(rmx, __shfl_xor(rmx, 32));
    const float na = norm_bound(rss, rmx, a.r);
    GridOut out[4];
#pragma unroll 1
    for (int jl = 0; jl < 4; ++jl) {
      // opaque copy of the sub-tile index: keeps the compiler from hoisting per-sub-tile
      // addresses and bounds of all four sub-tiles out of the round loop into registers
      int j = jl;
      asm volatile("" : "+s"(j));
      PhiRegs Pj = Pc[0];
      float nb = nbv[0];
      f32x4 acc[4];
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) acc[cb] = MULTI ? acc4[0][cb] : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 1; t < 4; ++t)
        if (j == t) {
          nb = nbv[t];
          Pj = Pc[t];
          if constexpr (MULTI) {
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) acc[cb] = acc4[t][cb];
          }
        }
      const int64_t c16 = cl0 + 16 * j;
      GridOut o;
      bool small = false;
      if constexpr (PACKED) {
        // integer Phi0: |delta| <= |c| ||A_i|| ||B_j|| below 1/2 on the whole sub-tile means
        // q = Phi0 (no rounding can move, nothing clips on a 4-bit grid)
        const float bound = fabsf(a.c) * na * nb * 1.02f;
        small = (B4 || a.bits == 4) && !__builtin_amdgcn_ballot_w64(!(bound < 0.5f - 0x1p-20f));
      }
      if (small) {
        grid_decide<PACKED, MASK, B4, Q8OUT>(a, Pj, acc, 0.f, false, row, c16, true, o);
      } else {
        if constexpr (!MULTI) {
#pragma unroll
          for (int cb = 0; cb < 4; ++cb) {
            const u32x4 ph = bfrag[j][0][cb][lane], pl = bfrag[j][1][cb][lane];
            acc[cb] = mfma16(ph, ah, acc[cb]);
            acc[cb] = mfma16(pl, ah, acc[cb]);
            acc[cb] = mfma16(ph, al, acc[cb]);
          }
        }
        // -1 where delta is exactly zero (a zero A row), so that no element is re-decided there
        const float tau = rmx == 0.f ? -1.f : a.tau_coef * na * nb;
        grid_decide<PACKED, MASK, B4, Q8OUT>(a, Pj, acc, tau, nb == 0.f, row, c16, false, o);
      }
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (j == t) out[t] = o;
    }
    // stores: the lane's 64 columns at once where they lie inside kq and are aligned
    const bool whole = row < a.m && cl0 + 64 <= a.kq;
    if constexpr (Q8OUT) {
      uint8_t* dst = a.qout + row * a.ldq + cl0;
      if (whole && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<u32x4*>(dst + 16 * j) = u32x4{out[j].qb[0], out[j].qb[1], out[j].qb[2], out[j].qb[3]};
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) grid_store<false, true>(a, out[j], row, cl0 + 16 * j);
      }
    } else {
      uint8_t* dst = a.qout + row * a.ldq + (cl0 >> 1);
      if (whole && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
          *reinterpret_cast<u32x4*>(dst + 16 * h) =
              u32x4{out[2 * h].w0, out[2 * h].w1, out[2 * h + 1].w0, out[2 * h + 1].w1};
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) grid_store<false, false>(a, out[j], row, cl0 + 16 * j);
      }
    }
    if constexpr (MASK) {
      uint16_t* md = a.mout + row * a.ldm + (cl0 >> 4);
      if (whole && (reinterpret_cast<uintptr_t>(md) & 7) == 0) {
        *reinterpret_cast<u32x2*>(md) =
            u32x2{(out[0].mb & 0xFFFFu) | (out[1].mb << 16), (out[2].mb & 0xFFFFu) | (out[3].mb << 16)};
      } else if (row < a.m) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (cl0 + 16 * j < a.kq) md[j] = uint16_t(out[j].mb);
      }
    }
  }
}

// ============================================================================ activations
// One block per token row: s_x = max|X_t| / 127, n = clip(round(X_t / s_x), -128, 127).
// Outputs (each optional): the codes n [T][ldn] (columns k..ldn-1 written as
// 0), X_hat = s_x n rounded to bfloat16 [T][ldh], and s_x [T].  VEC: k % 8 == 0
// and 16-byte aligned rows, read and written as 16-byte vectors.
template <bool VEC>
__global__ __launch_bounds__(256) void k_act_quant(const uint16_t* __restrict__ X, int64_t k,
                                                   int8_t* __restrict__ n, int64_t ldn,
                                                   uint16_t* __restrict__ xh, int64_t ldh,
                                                   float* __restrict__ sx) {
  const int64_t row = blockIdx.x;
  const uint16_t* x = X + row * k;
  float amax = 0.f;
  if (VEC) {
    for (int64_t j = 8 * threadIdx.x; j < k; j += 8 * 256) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(x + j);
#pragma unroll
      for (int q = 0; q < 4; ++q) amax = fmaxf(amax, fmaxf(fabsf(bf16_lo(v[q])), fabsf(bf16_hi(v[q]))));
    }
  } else {
    for (int64_t j = threadIdx.x; j < k; j += 256) amax = fmaxf(amax, fabsf(bf16_to_f32(x[j])));
  }
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  __shared__ float red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float s = amax / 127.f;
  if (threadIdx.x == 0 && sx) sx[row] = s;
  auto code = [&](float v) { return s > 0.f ? min(max(int(__builtin_rintf(v / s)), -128), 127) : 0; };
  if (VEC) {
    for (int64_t j = 8 * threadIdx.x; j < k; j += 8 * 256) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(x + j);
      int c[8];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c[2 * q] = code(bf16_lo(v[q]));
        c[2 * q + 1] = code(bf16_hi(v[q]));
      }
      if (n) {
        u32x2 o;
#pragma unroll
        for (int h = 0; h < 2; ++h)
          o[h] = uint32_t(c[4 * h] & 255) | (uint32_t(c[4 * h + 1] & 255) << 8) | (uint32_t(c[4 * h + 2] & 255) << 16) |
                 (uint32_t(c[4 * h + 3] & 255) << 24);
        *reinterpret_cast<u32x2*>(n + row * ldn + j) = o;
      }
      if (xh) {
        u32x4 o;
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = pack_bf16x2(float(c[2 * q]) * s, float(c[2 * q + 1]) * s);
        *reinterpret_cast<u32x4*>(xh + row * ldh + j) = o;
      }
    }
    if (n)
      for (int64_t j = k + threadIdx.x; j < ldn; j += 256) n[row * ldn + j] = 0;
  } else {
    const int64_t end = n ? ldn : k;
    for (int64_t j = threadIdx.x; j < end; j += 256) {
      const int c = j < k ? code(bf16_to_f32(x[j])) : 0;
      if (n) n[row * ldn + j] = int8_t(c);
      if (xh && j < k) xh[row * ldh + j] = __builtin_bit_cast(uint16_t, (__bf16)(float(c) * s));
    }
  }
}

// ============================================================================ launchers

hipError_t launch_minmax_scale(const float* W0, int64_t m, int64_t k, int64_t gsize, int bits, float* s0, int32_t* z0,
                               hipStream_t st) {
  const int ngroups = int(k / gsize);
  k_minmax_scale<<<unsigned(m * ngroups), 256, 0, st>>>(W0, k, gsize, ngroups, bits, s0, z0);
  return hipGetLastError();
}

hipError_t launch_encode(const float* W0, const float* s0, const int32_t* z0, int64_t m, int64_t k, int64_t gsize,
                         int bits, int packed, void* phi0, hipStream_t st) {
  const int64_t n = m * (packed ? k / 2 : k);
  const int ngroups = int(k / gsize);
  k_encode<<<unsigned((n + 255) / 256), 256, 0, st>>>(W0, s0, z0, m, k, gsize, ngroups, bits, packed, phi0);
  return hipGetLastError();
}

hipError_t launch_grid(const GridArgs& a0, hipStream_t st) {
  GridArgs a = a0;
  const int64_t nstrips = (a.kq + 4 * GR_COLS - 1) / (4 * GR_COLS), nrb = (a.m + 15) / 16;
  // 16-row rounds per wave: the most (up to 8) that still gives GR_MIN_BLOCKS blocks
  a.nit = 8;
  while (a.nit > 1 && nstrips * ((nrb + a.nit - 1) / a.nit) < GR_MIN_BLOCKS) a.nit /= 2;
  const int64_t nblocks = nstrips * ((nrb + a.nit - 1) / a.nit);
  a.tau_coef = float(1.02 * (3.0 * 0x1p-16 + (3.0 * a.r + 2.0) * 0x1p-23) * (a.c < 0 ? -a.c : a.c));
  const unsigned nb = unsigned(nblocks);
  const bool coal = a.r == 32 && a.k % 4 == 0 && (reinterpret_cast<uintptr_t>(a.A) & 15) == 0 &&
                    (reinterpret_cast<uintptr_t>(a.B) & 15) == 0;
  // 4-bit grids (the common W4 case) get an instantiation with the width fixed
  const int sel = (a.packed ? 8 : 0) | (a.r <= 32 ? 4 : 0) | (coal ? 2 : 0) | (a.mout ? 1 : 0);
  const bool b4 = a.bits == 4;
  // wide tiles (r a multiple of 32, 16-byte aligned rows) where they still give GRW_MIN_BLOCKS
  // blocks: rounds of 64 rows per block, the most (up to 4) that keep that many; r > 32
  // accumulates its rank chunks in one round per block
  const int64_t nrb64 = (a.m + 63) / 64;
  const bool phi16 = ((a.ld_phi | int64_t(reinterpret_cast<uintptr_t>(a.phi0))) & 15) == 0;
  const bool wide_ok = a.r % 32 == 0 && a.k % 4 == 0 && (reinterpret_cast<uintptr_t>(a.A) & 15) == 0 &&
                       (reinterpret_cast<uintptr_t>(a.B) & 15) == 0 && phi16;
  if (wide_ok && nstrips * nrb64 >= GRW_MIN_BLOCKS) {
    GridArgs w = a;
    const bool multi = a.r > 32;
    w.nit = multi ? 1 : 4;
    while (w.nit > 1 && nstrips * ((nrb64 + w.nit - 1) / w.nit) < GRW_MIN_BLOCKS) w.nit /= 2;
    const unsigned nbw = unsigned(nstrips * ((nrb64 + w.nit - 1) / w.nit));
    const int wsel = (multi ? 8 : 0) | (a.packed ? 4 : 0) | (a.mout ? 2 : 0) | (b4 ? 1 : 0);
    if (a.q8out) {
      if (a.packed || a.bits <= 4) return hipErrorInvalidValue;
      if (multi) {
        if (a.mout) k_grid_w<false, true, false, true, true><<<nbw, GR_THREADS, 0, st>>>(w);
        else k_grid_w<false, false, false, true, true><<<nbw, GR_THREADS, 0, st>>>(w);
      } else {
        if (a.mout) k_grid_w<false, true, false, true, false><<<nbw, GR_THREADS, 0, st>>>(w);
        else k_grid_w<false, false, false, true, false><<<nbw, GR_THREADS, 0, st>>>(w);
      }
      return hipGetLastError();
    }
    switch (wsel) {
#define LRQAT_GRIDW_CASE(S, P, M, B, U)                                     \
  case S:                                                                   \
    k_grid_w<P, M, B, false, U><<<nbw, GR_THREADS, 0, st>>>(w);             \
    break;
      LRQAT_GRIDW_CASE(0, false, false, false, false)
      LRQAT_GRIDW_CASE(1, false, false, true, false)
      LRQAT_GRIDW_CASE(2, false, true, false, false)
      LRQAT_GRIDW_CASE(3, false, true, true, false)
      LRQAT_GRIDW_CASE(4, true, false, false, false)
      LRQAT_GRIDW_CASE(5, true, false, true, false)
      LRQAT_GRIDW_CASE(6, true, true, false, false)
      LRQAT_GRIDW_CASE(7, true, true, true, false)
      LRQAT_GRIDW_CASE(8, false, false, false, true)
      LRQAT_GRIDW_CASE(9, false, false, true, true)
      LRQAT_GRIDW_CASE(10, false, true, false, true)
      LRQAT_GRIDW_CASE(11, false, true, true, true)
      LRQAT_GRIDW_CASE(12, true, false, false, true)
      LRQAT_GRIDW_CASE(13, true, false, true, true)
      LRQAT_GRIDW_CASE(14, true, true, false, true)
      LRQAT_GRIDW_CASE(15, true, true, true, true)
#undef LRQAT_GRIDW_CASE
    }
    return hipGetLastError();
  }
  // grids wider than 4 bits (fixed point b = 5..7) are written as int8
  if (a.q8out) {
    if (a.packed || a.bits <= 4) return hipErrorInvalidValue;
    switch (sel) {
#define LRQAT_GRID8_CASE(S, O, C, M)                                        \
  case S:                                                                   \
    k_grid<false, O, M, C, false, true><<<nb, GR_THREADS, 0, st>>>(a);      \
    break;
      LRQAT_GRID8_CASE(0, false, false, false)
      LRQAT_GRID8_CASE(1, false, false, true)
      LRQAT_GRID8_CASE(4, true, false, false)
      LRQAT_GRID8_CASE(5, true, false, true)
      LRQAT_GRID8_CASE(6, true, true, false)
      LRQAT_GRID8_CASE(7, true, true, true)
#undef LRQAT_GRID8_CASE
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  switch (sel) {
#define LRQAT_GRID_CASE(S, P, O, C, M)                                      \
  case S:                                                                   \
    if (b4) k_grid<P, O, M, C, true, false><<<nb, GR_THREADS, 0, st>>>(a);  \
    else k_grid<P, O, M, C, false, false><<<nb, GR_THREADS, 0, st>>>(a);    \
    break;
    LRQAT_GRID_CASE(0, false, false, false, false)
    LRQAT_GRID_CASE(1, false, false, false, true)
    LRQAT_GRID_CASE(4, false, true, false, false)
    LRQAT_GRID_CASE(5, false, true, false, true)
    LRQAT_GRID_CASE(6, false, true, true, false)
    LRQAT_GRID_CASE(7, false, true, true, true)
    LRQAT_GRID_CASE(8, true, false, false, false)
    LRQAT_GRID_CASE(9, true, false, false, true)
    LRQAT_GRID_CASE(12, true, true, false, false)
    LRQAT_GRID_CASE(13, true, true, false, true)
    LRQAT_GRID_CASE(14, true, true, true, false)
    LRQAT_GRID_CASE(15, true, true, true, true)
#undef LRQAT_GRID_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_act_quant(const uint16_t* X, int64_t T, int64_t k, int8_t* n, int64_t ldn, uint16_t* xh, int64_t ldh,
                            float* sx, hipStream_t st) {
  if (T == 0) return hipSuccess;
  const bool vec = k % 8 == 0 && (reinterpret_cast<uintptr_t>(X) & 15) == 0 && (!n || ldn % 8 == 0) &&
                   (!xh || (ldh % 8 == 0 && (reinterpret_cast<uintptr_t>(xh) & 15) == 0)) &&
                   (reinterpret_cast<uintptr_t>(n) & 7) == 0;
  if (vec) k_act_quant<true><<<unsigned(T), 256, 0, st>>>(X, k, n, ldn, xh, ldh, sx);
  else k_act_quant<false><<<unsigned(T), 256, 0, st>>>(X, k, n, ldn, xh, ldh, sx);
  return hipGetLastError();
}

}  // namespace lrqat
