// bf16 MFMA GEMMs of the LR-QAT layer on gfx950.
//
//   kFwd  Y  = X_hat W_hat^T      M = T, N = m, K = k   (Section 3, Eq. lr_qat)
//   kDx   dX = dY W_hat           M = T, N = k, K = m
//   kDw   dW = dY^T X_hat         M = m, N = k, K = T, never stored: the
//         epilogue forms G = s * M * dW and the rank-r partial products
//         G B^T and A^T G (Section 3, STE gradients w.r.t. A and B).
//
// W_hat enters as the integer grid q written by the grid pass (packed int4, or
// int8 for grids of 5..7 bits); the operand loaders unpack it into bfloat16
// tiles in LDS (q - z is exact in bfloat16 for |q - z| <= 256), with the scale
// s applied in the epilogue (forward, per channel) or folded into the tile
// (dX, and the forward with group-wise scales).
//
// Block tile 256 x 256 x 64, four waves in a 2 x 2 arrangement, each wave a
// 128 x 128 sub-tile of 4 x 4 MFMA 32x32x16 blocks.  Two LDS stages of
// (256 + 256) x 64 bfloat16 (128 KiB); the next K-tile is fetched into
// registers while the current one feeds the MFMAs.  The forward and dX output
// tiles leave through LDS as whole row segments.
#pragma once

#include "kernels.h"

namespace lrqat {

constexpr int BM = GEMM_BM, BN = GEMM_BN, BK = GEMM_BK;
// Operand tiles in LDS are [256 rows][64] bfloat16 (128-byte rows of eight
// 16-byte chunks).  Chunk c of row r sits at chunk slot c ^ g(r) with
// g(r) = (r & 7) ^ ((r >> 3) & 1): any 8 consecutive rows read at one chunk
// hit 8 different slots (32 banks), any 16 consecutive rows hit 16 different
// (row parity, slot) pairs (64 banks).  g depends on r mod 16 only, so the
// fragments of row blocks 32 apart are constant offsets of one address.
constexpr int TILE = 256 * 64;  // elements of one operand tile
__device__ __forceinline__ int tile_g(int row) { return (row & 7) ^ ((row >> 3) & 1); }
__device__ __forceinline__ int tile_off(int row, int chunk) { return row * 64 + ((chunk ^ tile_g(row)) << 3); }

// ------------------------------------------------------------------ buffer resources
// Operands are read with raw buffer loads.  A load whose per-lane offset is
// at or past the resource's num_records returns zeros, so a tile that
// overhangs the end of a tensor needs no per-lane branch: each resource
// starts at the tile's origin and all strides stay in the per-lane offset.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, int64_t bytes) {
  const int64_t n = bytes < 0 ? 0 : (bytes > int64_t(0xFFFFFFFF) ? int64_t(0xFFFFFFFF) : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), short(0), int(uint32_t(n)), 0x00020000);
}
__device__ __forceinline__ u32x4 ld128(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, int(off), 0, 0));
}
__device__ __forceinline__ u32x2 ld64(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, int(off), 0, 0));
}
__device__ __forceinline__ uint32_t ld32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, int(off), 0, 0);
}
__device__ __forceinline__ uint32_t ld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, int(off), 0, 0);
}
__device__ __forceinline__ float ldf(__amdgpu_buffer_rsrc_t r, uint32_t off) { return __uint_as_float(ld32(r, off)); }

// 8 bfloat16 starting at byte offset `off` with 16-bit loads (rows not 16-byte aligned).
__device__ __forceinline__ u32x4 ld8_bf16_scalar(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  u32x4 v;
#pragma unroll
  for (int q = 0; q < 4; ++q) v[q] = ld16(r, off + 4 * q) | (ld16(r, off + 4 * q + 2) << 16);
  return v;
}

// Zero the elements of an 8-wide bfloat16 chunk at column kk that lie at or past K.
__device__ __forceinline__ u32x4 mask_tail(u32x4 v, int kk, int K) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t lo = (kk + 2 * q < K) ? 0x0000FFFFu : 0u, hi = (kk + 2 * q + 1 < K) ? 0xFFFF0000u : 0u;
    v[q] &= lo | hi;
  }
  return v;
}

// ------------------------------------------------------------------ K-contiguous bf16 source
// 256 x 64 tile of a row-major [rows][K] bfloat16 matrix (forward X, dX's dY);
// thread t loads chunk t%8 of rows t/8 + 32 i.
struct RegsKc {
  u32x4 v[8];
  int kk;      // first column of the thread's chunk (columns >= K are masked on the generic path)
};

template <bool VEC>
__device__ __forceinline__ void load_kc_bf16(RegsKc& R, const uint16_t* __restrict__ src, int64_t ld,
                                             int64_t row0, int64_t nrows, int64_t k0, int64_t K) {
  const int t = threadIdx.x;
  const auto r = rsrc(src + row0 * ld, (nrows - row0) * ld * 2);
  R.kk = int(k0) + 8 * (t & 7);
  const uint32_t base = uint32_t(((t >> 3) * ld + R.kk) * 2), step = uint32_t(32 * ld * 2);
#pragma unroll
  for (int i = 0; i < 8; ++i) R.v[i] = VEC ? ld128(r, base + i * step) : ld8_bf16_scalar(r, base + i * step);
}

// Each operand tile is written to LDS as 8 16-byte stores per thread; the
// *_one functions do store number w (0..7), so the main loop can spread them
// between MFMA groups.
template <bool VEC>
__device__ __forceinline__ void store_kc_one(uint16_t* tile, const RegsKc& R, int64_t K, int i) {
  const int t = threadIdx.x;
  u32x4 v = R.v[i];
  if (!VEC) v = mask_tail(v, R.kk, int(K));
  *reinterpret_cast<u32x4*>(tile + tile_off((t >> 3) + 32 * i, t & 7)) = v;
}

// ------------------------------------------------------------------ K-contiguous int8 source (W4A8 codes)
// n [T][ld] is zero beyond column k, so no K mask is needed.
struct RegsKc8 {
  u32x2 v[8];
};

__device__ __forceinline__ void load_kc_i8(RegsKc8& R, const int8_t* __restrict__ src, int64_t ld,
                                           int64_t row0, int64_t nrows, int64_t k0) {
  const int t = threadIdx.x;
  const auto r = rsrc(src + row0 * ld, (nrows - row0) * ld);
  const uint32_t base = uint32_t((t >> 3) * ld + k0 + 8 * (t & 7)), step = uint32_t(32 * ld);
#pragma unroll
  for (int i = 0; i < 8; ++i) R.v[i] = ld64(r, base + i * step);
}

__device__ __forceinline__ void store_kc_i8_one(uint16_t* tile, const RegsKc8& R, int i) {
  const int t = threadIdx.x;
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t w = R.v[i][q >> 1];
    o[q] = pack_bf16x2(float(sbyte(w, 2 * (q & 1))), float(sbyte(w, 2 * (q & 1) + 1)));
  }
  *reinterpret_cast<u32x4*>(tile + tile_off((t >> 3) + 32 * i, t & 7)) = o;
}

// ------------------------------------------------------------------ zero offsets
// z[row][grp] (z shaped like s; grp = 0 for one offset per row) as an int;
// rows past the end read 0.
__device__ __forceinline__ int ld_z(__amdgpu_buffer_rsrc_t rz, int64_t idx) { return int(ld32(rz, uint32_t(idx * 4))); }

// ------------------------------------------------------------------ packed q, K-contiguous (forward B)
// 256 weight rows x 64 K-values = 256 x 32 bytes; thread t takes 16 bytes
// (32 values) of rows t/2 and t/2 + 128.  q is zero past column k.
struct RegsQKc {
  u32x4 v[2];
  float sc[2];
  int zi[2];
};

template <bool GRP, bool ZP>
__device__ __forceinline__ void load_q_kc(RegsQKc& R, const GemmArgs& p, int64_t row0, int64_t k0) {
  const int t = threadIdx.x;
  const int64_t kk = k0 + 32 * (t & 1);
  const auto rq = rsrc(static_cast<const uint8_t*>(p.b) + row0 * p.ldb, (p.N - row0) * p.ldb);
  const uint32_t base = uint32_t((t >> 1) * p.ldb + (kk >> 1)), step = uint32_t(128 * p.ldb);
#pragma unroll
  for (int i = 0; i < 2; ++i) R.v[i] = ld128(rq, base + i * step);
  const int64_t grp = GRP ? kk / p.gsize : 0;
  if (GRP) {
    const auto rs = rsrc(p.s + row0 * p.ngroups, (p.N - row0) * p.ngroups * 4);
    const uint32_t sb = uint32_t(((t >> 1) * p.ngroups + grp) * 4), sstep = uint32_t(128 * p.ngroups * 4);
#pragma unroll
    for (int i = 0; i < 2; ++i) R.sc[i] = ldf(rs, sb + i * sstep);
  }
  if (ZP) {
    const auto rz = rsrc(p.z + row0 * p.ngroups, (p.N - row0) * p.ngroups * 4);
#pragma unroll
    for (int i = 0; i < 2; ++i) R.zi[i] = ld_z(rz, ((t >> 1) + 128 * i) * p.ngroups + grp);
  }
}

template <bool GRP, bool ZP>
__device__ __forceinline__ void store_q_kc_one(uint16_t* tile, const RegsQKc& R, int w8) {
  const int t = threadIdx.x;
  const int i = w8 >> 2, c = w8 & 3;  // row half, 16-byte chunk
  const int row = (t >> 1) + 128 * i;
  const uint32_t w = R.v[i][c];
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    int na = nibble(w, 2 * q), nb = nibble(w, 2 * q + 1);
    if (ZP) {
      na -= R.zi[i];
      nb -= R.zi[i];
    }
    float a = float(na), b = float(nb);
    if (GRP) {
      a *= R.sc[i];
      b *= R.sc[i];
    }
    o[q] = pack_bf16x2(a, b);
  }
  *reinterpret_cast<u32x4*>(tile + tile_off(row, 4 * (t & 1) + c)) = o;
}

// ------------------------------------------------------------------ int8 q, K-contiguous (forward B, 5..7-bit grids)
// 256 weight rows x 64 bytes: thread t loads 8 bytes of rows t/8 + 32 i; q is zero past column k.
struct RegsQKc8 {
  u32x2 v[8];
  float sc[8];
  int zi[8];
};

template <bool GRP, bool ZP>
__device__ __forceinline__ void load_q_kc8(RegsQKc8& R, const GemmArgs& p, int64_t row0, int64_t k0) {
  const int t = threadIdx.x;
  const auto rq = rsrc(static_cast<const uint8_t*>(p.b) + row0 * p.ldb, (p.N - row0) * p.ldb);
  const int64_t kk = k0 + 8 * (t & 7);
  const uint32_t base = uint32_t((t >> 3) * p.ldb + kk), step = uint32_t(32 * p.ldb);
#pragma unroll
  for (int i = 0; i < 8; ++i) R.v[i] = ld64(rq, base + i * step);
  const int64_t grp = GRP ? kk / p.gsize : 0;
  if (GRP) {
    const auto rs = rsrc(p.s + row0 * p.ngroups, (p.N - row0) * p.ngroups * 4);
#pragma unroll
    for (int i = 0; i < 8; ++i) R.sc[i] = ldf(rs, uint32_t((((t >> 3) + 32 * i) * p.ngroups + grp) * 4));
  }
  if (ZP) {
    const auto rz = rsrc(p.z + row0 * p.ngroups, (p.N - row0) * p.ngroups * 4);
#pragma unroll
    for (int i = 0; i < 8; ++i) R.zi[i] = ld_z(rz, ((t >> 3) + 32 * i) * p.ngroups + grp);
  }
}

template <bool GRP, bool ZP>
__device__ __forceinline__ void store_q_kc8_one(uint16_t* tile, const RegsQKc8& R, int i) {
  const int t = threadIdx.x;
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t w = R.v[i][q >> 1];
    int na = sbyte(w, 2 * (q & 1)), nb = sbyte(w, 2 * (q & 1) + 1);
    if (ZP) {
      na -= R.zi[i];
      nb -= R.zi[i];
    }
    float a = float(na), b = float(nb);
    if (GRP) {
      a *= R.sc[i];
      b *= R.sc[i];
    }
    o[q] = pack_bf16x2(a, b);
  }
  *reinterpret_cast<u32x4*>(tile + tile_off((t >> 3) + 32 * i, t & 7)) = o;
}

// ------------------------------------------------------------------ K-strided sources
// Tile rows are the index contiguous in memory, K the strided one.  Thread t
// covers 8 consecutive tile rows 8 (t/8) .. +7 (one vector per K-line) of
// the 8 K-lines 8 (t%8) .. +7 and transposes them in registers into 8
// chunks; the 8 lanes of a K-group fill one 128-byte row segment of LDS.
// Columns past a tensor's width only feed output rows/columns that the
// epilogue discards; K-lines past the end read as zeros.

// packed q (dX B): K = weight rows (m), tile rows = weight columns (k).
// Values are scaled by their row's (or row-group's) s before rounding to bf16.
struct RegsQKs {
  uint32_t w[8];
  float sc[8];
  int zi[8];
};

// Scales (and zero offsets) of the 8 K-lines (weight rows) k0 + 8 kg .. +7 at column col.
template <bool GRP, bool ZP>
__device__ __forceinline__ void load_ks_scales(float (&sc)[8], int (&zi)[8], const GemmArgs& p, int64_t k0, int kg,
                                               int64_t col) {
  const int64_t grp = GRP ? col / p.gsize : 0;
  if (GRP) {
    const auto rs = rsrc(p.s + k0 * p.ngroups, (p.K - k0) * p.ngroups * 4);
    const uint32_t sb = uint32_t((8 * kg * p.ngroups + grp) * 4), sstep = uint32_t(p.ngroups * 4);
#pragma unroll
    for (int e = 0; e < 8; ++e) sc[e] = ldf(rs, sb + e * sstep);
  } else {
    // the 8 rows' scales are consecutive: two 16-byte loads (rows past K read as zeros)
    const auto rs = rsrc(p.s + k0, (p.K - k0) * 4);
    const u32x4 s0 = ld128(rs, uint32_t(8 * kg * 4)), s1 = ld128(rs, uint32_t((8 * kg + 4) * 4));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      sc[e] = __uint_as_float(s0[e]);
      sc[4 + e] = __uint_as_float(s1[e]);
    }
  }
  if (ZP) {
    const auto rz = rsrc(p.z + k0 * p.ngroups, (p.K - k0) * p.ngroups * 4);
#pragma unroll
    for (int e = 0; e < 8; ++e) zi[e] = ld_z(rz, (8 * kg + e) * p.ngroups + grp);
  }
}

template <bool GRP, bool ZP>
__device__ __forceinline__ void load_q_ks(RegsQKs& R, const GemmArgs& p, int64_t n0, int64_t k0) {
  const int t = threadIdx.x;
  const int kg = t & 7, a = t >> 3;
  const int64_t col = n0 + 8 * a;
  const auto rq = rsrc(static_cast<const uint8_t*>(p.b) + k0 * p.ldb, (p.K - k0) * p.ldb);
  const uint32_t base = uint32_t(8 * kg * p.ldb + (col >> 1)), step = uint32_t(p.ldb);
#pragma unroll
  for (int e = 0; e < 8; ++e) R.w[e] = ld32(rq, base + e * step);
  load_ks_scales<GRP, ZP>(R.sc, R.zi, p, k0, kg, col);
}

template <bool ZP>
__device__ __forceinline__ void store_q_ks_one(uint16_t* tile, const RegsQKs& R, int c) {
  const int t = threadIdx.x;
  const int kg = t & 7, a = t >> 3;
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    int na = nibble(R.w[2 * q], c), nb = nibble(R.w[2 * q + 1], c);
    if (ZP) {
      na -= R.zi[2 * q];
      nb -= R.zi[2 * q + 1];
    }
    o[q] = pack_bf16x2(float(na) * R.sc[2 * q], float(nb) * R.sc[2 * q + 1]);
  }
  *reinterpret_cast<u32x4*>(tile + tile_off(8 * a + c, kg)) = o;
}

// int8 q (dX B, 5..7-bit grids): 8 bytes (columns 8a .. 8a + 7) of each K-line.
struct RegsQKs8 {
  u32x2 v[8];
  float sc[8];
  int zi[8];
};

template <bool GRP, bool ZP>
__device__ __forceinline__ void load_q_ks8(RegsQKs8& R, const GemmArgs& p, int64_t n0, int64_t k0) {
  const int t = threadIdx.x;
  const int kg = t & 7, a = t >> 3;
  const int64_t col = n0 + 8 * a;
  const auto rq = rsrc(static_cast<const uint8_t*>(p.b) + k0 * p.ldb, (p.K - k0) * p.ldb);
  const uint32_t base = uint32_t(8 * kg * p.ldb + col), step = uint32_t(p.ldb);
#pragma unroll
  for (int e = 0; e < 8; ++e) R.v[e] = ld64(rq, base + e * step);
  load_ks_scales<GRP, ZP>(R.sc, R.zi, p, k0, kg, col);
}

template <bool ZP>
__device__ __forceinline__ void store_q_ks8_one(uint16_t* tile, const RegsQKs8& R, int c) {
  const int t = threadIdx.x;
  const int kg = t & 7, a = t >> 3;
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    int na = sbyte(R.v[2 * q][c >> 2], c & 3), nb = sbyte(R.v[2 * q + 1][c >> 2], c & 3);
    if (ZP) {
      na -= R.zi[2 * q];
      nb -= R.zi[2 * q + 1];
    }
    o[q] = pack_bf16x2(float(na) * R.sc[2 * q], float(nb) * R.sc[2 * q + 1]);
  }
  *reinterpret_cast<u32x4*>(tile + tile_off(8 * a + c, kg)) = o;
}

// bfloat16 (dW A = dY, dW B = X): 16-byte vector per K-line.
struct RegsKs {
  u32x4 v[8];
};

template <bool VEC>
__device__ __forceinline__ void load_ks_bf16(RegsKs& R, const uint16_t* __restrict__ src, int64_t ld,
                                             int64_t c0, int64_t k0, int64_t K) {
  const int t = threadIdx.x;
  const int kg = t & 7, a = t >> 3;
  const auto r = rsrc(src + k0 * ld + c0, (K - k0) * ld * 2 - c0 * 2);
  const uint32_t base = uint32_t((8 * kg * ld + 8 * a) * 2), step = uint32_t(ld * 2);
#pragma unroll
  for (int e = 0; e < 8; ++e) R.v[e] = VEC ? ld128(r, base + e * step) : ld8_bf16_scalar(r, base + e * step);
}

__device__ __forceinline__ void store_ks_bf16_one(uint16_t* tile, const RegsKs& R, int c) {
  const int t = threadIdx.x;
  const int kg = t & 7, a = t >> 3;
  u32x4 o;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t x = R.v[2 * q][c >> 1], y = R.v[2 * q + 1][c >> 1];
    o[q] = (c & 1) ? perm_hi16(x, y) : perm_lo16(x, y);
  }
  *reinterpret_cast<u32x4*>(tile + tile_off(8 * a + c, kg)) = o;
}

// ------------------------------------------------------------------ the kernel

template <int V, bool ACT, bool GRP, bool VEC, int OPT>
struct Loader;

// store_one(w): LDS store w of the tile held in registers, w = 0..7 for the A
// operand and 8..15 for the B operand.
template <bool ACT, bool GRP, bool VEC, int OPT>
struct Loader<kFwd, ACT, GRP, VEC, OPT> {
  static constexpr bool ZP = (OPT & kOptZ) != 0, Q8 = (OPT & kOptQ8) != 0;
  typename std::conditional<ACT, RegsKc8, RegsKc>::type ra;
  typename std::conditional<Q8, RegsQKc8, RegsQKc>::type rb;
  __device__ __forceinline__ void load(const GemmArgs& p, int64_t m0, int64_t n0, int64_t k0) {
    if constexpr (ACT) load_kc_i8(ra, static_cast<const int8_t*>(p.a), p.lda, m0, p.M, k0);
    else load_kc_bf16<VEC>(ra, static_cast<const uint16_t*>(p.a), p.lda, m0, p.M, k0, p.K);
    if constexpr (Q8) load_q_kc8<GRP, ZP>(rb, p, n0, k0);
    else load_q_kc<GRP, ZP>(rb, p, n0, k0);
  }
  __device__ __forceinline__ void store_one(const GemmArgs& p, uint16_t* As, uint16_t* Bs, int w) {
    if (w < 8) {
      if constexpr (ACT) store_kc_i8_one(As, ra, w);
      else store_kc_one<VEC>(As, ra, p.K, w);
    } else {
      if constexpr (Q8) store_q_kc8_one<GRP, ZP>(Bs, rb, w - 8);
      else store_q_kc_one<GRP, ZP>(Bs, rb, w - 8);
    }
  }
};

template <bool ACT, bool GRP, bool VEC, int OPT>
struct Loader<kDx, ACT, GRP, VEC, OPT> {
  static constexpr bool ZP = (OPT & kOptZ) != 0, Q8 = (OPT & kOptQ8) != 0;
  RegsKc ra;
  typename std::conditional<Q8, RegsQKs8, RegsQKs>::type rb;
  __device__ __forceinline__ void load(const GemmArgs& p, int64_t m0, int64_t n0, int64_t k0) {
    load_kc_bf16<VEC>(ra, static_cast<const uint16_t*>(p.a), p.lda, m0, p.M, k0, p.K);
    if constexpr (Q8) load_q_ks8<GRP, ZP>(rb, p, n0, k0);
    else load_q_ks<GRP, ZP>(rb, p, n0, k0);
  }
  __device__ __forceinline__ void store_one(const GemmArgs& p, uint16_t* As, uint16_t* Bs, int w) {
    if (w < 8) {
      store_kc_one<VEC>(As, ra, p.K, w);
    } else {
      if constexpr (Q8) store_q_ks8_one<ZP>(Bs, rb, w - 8);
      else store_q_ks_one<ZP>(Bs, rb, w - 8);
    }
  }
};

template <bool ACT, bool GRP, bool VEC, int OPT>
struct Loader<kDw, ACT, GRP, VEC, OPT> {
  static_assert(!ACT, "the dW GEMM reads bfloat16 operands (W4A8: X_hat)");
  RegsKs ra, rb;
  __device__ __forceinline__ void load(const GemmArgs& p, int64_t m0, int64_t n0, int64_t k0) {
    load_ks_bf16<VEC>(ra, static_cast<const uint16_t*>(p.a), p.lda, m0, k0, p.K);
    load_ks_bf16<VEC>(rb, static_cast<const uint16_t*>(p.b), p.ldb, n0, k0, p.K);
  }
  __device__ __forceinline__ void store_one(const GemmArgs&, uint16_t* As, uint16_t* Bs, int w) {
    if (w < 8) store_ks_bf16_one(As, ra, w);
    else store_ks_bf16_one(Bs, rb, w - 8);
  }
};

// Offset of element (i, j) in a [rows][256] bfloat16 staging tile of an
// epilogue (the output tile; dW's G and its A/B blocks): the 32 16-byte chunks of a 512-byte row are
// permuted by i mod 32, so 32 consecutive rows read at one column hit 32
// different chunk slots.
__device__ __forceinline__ int g_off(int i, int j) { return i * 256 + ((((j >> 3) ^ (i & 31))) << 3) + (j & 7); }

// LDS transpose load (gfx950): lane i of each 16-lane group receives the 4
// values in column i % 4 of the 4-element rows that lanes 4 e + i / 4 address
// (e = 0..3).
typedef short s16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x2 ld_tr16(const uint16_t* p) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(const_cast<uint16_t*>(p)));
  return __builtin_bit_cast(u32x2, v);
}

// MFMA operand from a [K][256] staging tile laid out by g_off: lane l gets
// column c0 + l % 32 at the 8 K rows k0 + 8 (l / 32) .. +7.  Lanes 4 e + q of
// each 16-lane group point at K row k0 + 8 (l / 32) + e (+4 for the second
// half) and columns c0 + 16 ((l / 16) % 2) + 4 q, so lane i of the group
// receives column c0 + 16 ((l / 16) % 2) + i.
__device__ __forceinline__ u32x4 frag_tr_g(const uint16_t* tile, int c0, int k0, int lane) {
  const int g = lane >> 4, r = lane & 15;
  const int c = c0 + 16 * (g & 1) + 4 * (r & 3);
  const int k = k0 + 8 * (g >> 1) + (r >> 2);
  const u32x2 lo = ld_tr16(tile + g_off(k, c));
  const u32x2 hi = ld_tr16(tile + g_off(k + 4, c));
  return u32x4{lo[0], lo[1], hi[0], hi[1]};
}

// Instruction interleave of one k-step (16 MFMAs, one scheduling region
// closed by a sched_barrier): each MFMA is followed by a few VALU ops of the
// next tile's conversion; the 8 fragment reads of the following k-step ride on
// the first MFMAs, the LDS stores of the next tile and the global loads of
// the tile after it are spread over the sequence.
enum : int { SG_VALU = 0x2, SG_MFMA = 0x8, SG_VMEM_READ = 0x20, SG_DS_READ = 0x100, SG_DS_WRITE = 0x200 };

// Schedules of the main loop, per GEMM, chosen by timing variants against
// each other on the 4096 x 4096, T = 8192 layer (same process, interleaved
// repeats): the pipeline, the k-step that issues the next tile's global loads,
// and for one k-step the VALU ops after each MFMA, LDS stores per pair of
// MFMAs and global loads per MFMA.  Against the single-region loop with the
// barrier at the end of the tile: forward -5.5%, dX -8%, dW -2%.
enum : int { kPipeSpread = 0, kPipeOneSet = 1, kPipeTile = 2 };
template <int V>
struct Sched {
  static constexpr int kPipe = kPipeSpread;
  static constexpr int kLoadStep = 1;
  static constexpr int kValu = V == kFwd ? 4 : 3;
  static constexpr int kWritesPerPair = 1;
  static constexpr int kVmemPerMfma = 1;
};

template <class S, bool VMEM, bool WRITES>
__device__ __forceinline__ void interleave_kstep() {
#pragma unroll
  for (int m = 0; m < 16; ++m) {
    __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
    if (m < 8) __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
    __builtin_amdgcn_sched_group_barrier(SG_VALU, S::kValu, 0);
    if (WRITES && (m & 1)) __builtin_amdgcn_sched_group_barrier(SG_DS_WRITE, S::kWritesPerPair, 0);
    if (VMEM) __builtin_amdgcn_sched_group_barrier(SG_VMEM_READ, S::kVmemPerMfma, 0);
  }
}

// The whole-tile region: the first k-step's fragment reads, then each MFMA
// followed by a few VALU ops of the next tile's conversion; the following
// k-steps' reads ride on the first MFMAs of each k-step, the LDS stores of the
// next tile and the global loads of the tile after it spread over the sequence.
__device__ __forceinline__ void interleave_tile() {
  __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 8, 0);
#pragma unroll
  for (int m = 0; m < 64; ++m) {
    __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
    __builtin_amdgcn_sched_group_barrier(SG_VALU, 3, 0);
    if ((m & 15) < 8 && m < 48) __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
    if ((m & 3) == 3) __builtin_amdgcn_sched_group_barrier(SG_DS_WRITE, 1, 0);
    if ((m & 3) == 1) __builtin_amdgcn_sched_group_barrier(SG_VMEM_READ, 1, 0);
  }
}

// The k-step after the barrier: the next tile's first 8 fragment reads first,
// then the 16 MFMAs of this tile's last k-step.
__device__ __forceinline__ void interleave_last() {
  __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 8, 0);
  __builtin_amdgcn_sched_group_barrier(SG_MFMA, 16, 0);
}

// Block -> tile order.  Blocks are dealt round-robin to the 8 XCDs (each with
// its own L2), so block b is renumbered to v = (b % 8) * (nt / 8) + b / 8: the
// blocks an XCD runs get consecutive numbers.  v then walks the tiles in
// groups of 4 tile rows (all columns of a group before the next group), so an
// XCD's concurrent blocks cover a compact 4 x 8 patch of tiles and share
// operand strips in its L2.
__device__ __forceinline__ void tile_of(int64_t b, int64_t ntm, int64_t ntn, int64_t& tm, int64_t& tn) {
  const int64_t nt = ntm * ntn, per = nt / 8;
  const int64_t v = b < per * 8 ? (b % 8) * per + b / 8 : b;
  constexpr int64_t GM = 4;
  const int64_t gsz = GM * ntn;
  const int64_t first = (v / gsz) * GM;
  const int64_t gm = ntm - first < GM ? ntm - first : GM;
  const int64_t off = v % gsz;
  tm = first + off % gm;
  tn = off / gm;
}

template <int V, bool ACT, bool GRP, bool VEC, int OPT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_gemm(GemmArgs p) {
  // A stages 0, 1 then B stages 0, 1 (128 KiB); the dW epilogue reuses all
  // of it for G.
  __shared__ __attribute__((aligned(16))) uint16_t lds[4 * TILE];
  __shared__ float s_tile[256];                                     // dW epilogue: per-channel scales
  __shared__ __attribute__((aligned(16))) uint16_t rt_tile[32 * 256];  // dW epilogue: A or B rank block (bf16)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t ntm = (p.M + BM - 1) / BM;
  int64_t tm, tn;
  tile_of(int64_t(blockIdx.x), ntm, (p.N + BN - 1) / BN, tm, tn);
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int wm = (wave >> 1) * 128, wn = (wave & 1) * 128;

  f32x16 acc[4][4];
  #pragma unroll
  for (int a = 0; a < 4; ++a)
    #pragma unroll
    for (int b = 0; b < 4; ++b)
      #pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;

  // Software pipeline over K-tiles of 64.  While the MFMAs consume LDS stage
  // kt%2, the registers holding tile kt+1 are written to the other stage and
  // the tile kt+2 is fetched.  kPipe picks the schedule (per GEMM, measured):
  //  * kPipeSpread: two register sets; the 16 stores of tile kt+1 spread over
  //    k-steps 0..2 while tile kt+2 loads into the other set from k-step
  //    kLoadStep on;
  //  * kPipeOneSet: one register set; the 16 stores in k-step 0, the reload
  //    with tile kt+2 in k-step 1;
  //  * kPipeTile: two register sets, the whole tile one scheduling region
  //    (stores after the MFMAs), the barrier at its end.
  // In the first two the one barrier per tile sits before k-step 3, whose
  // fragments are already in registers, so the first fragments of tile kt+1
  // are read right after it and their latency hides behind k-step 3's MFMAs.
  // Loads past the last tile read zeros or unused data and are never
  // consumed, so the body has no branches.
  using Ld = Loader<V, ACT, GRP, VEC, OPT>;
  using S = Sched<V>;
  const int nk = int((p.K + BK - 1) / BK);
  u32x4 fa[2][4], fb[2][4];
  auto read = [&](u32x4 (&a)[4], u32x4 (&b)[4], const uint16_t* As, const uint16_t* Bs, int s) {
    const int ch = 2 * s + (lane >> 5);
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = *reinterpret_cast<const u32x4*>(As + tile_off(wm + 32 * i + (lane & 31), ch));
#pragma unroll
    for (int j = 0; j < 4; ++j) b[j] = *reinterpret_cast<const u32x4*>(Bs + tile_off(wn + 32 * j + (lane & 31), ch));
  };
  auto mfmas = [&](const u32x4 (&a)[4], const u32x4 (&b)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        // D = B-tile x A-tile^T: a lane's accumulator holds 4 consecutive output
        // columns of one output row (8-byte stores; dW: 4 columns of one weight row)
        acc[i][j] = mfma32(b[j], a[i], acc[i][j]);
  };
  // order of a tile's 16 LDS stores (A: 0..7, B: 8..15), alternating operands
  constexpr int kOrder[16] = {0, 8, 1, 9, 2, 10, 3, 11, 4, 12, 5, 13, 6, 14, 7, 15};
  // the last k-step of tile kt (after the barrier) with the first fragment reads of tile kt+1
  auto last_kstep = [&](const uint16_t* Asn, const uint16_t* Bsn) {
    __syncthreads();
    read(fa[0], fb[0], Asn, Bsn, 0);
    mfmas(fa[1], fb[1]);
    interleave_last();
    __builtin_amdgcn_sched_barrier(0);
  };

  if constexpr (S::kPipe == kPipeSpread) {
    Ld L0, L1;
    L0.load(p, m0, n0, 0);
    L1.load(p, m0, n0, BK);
#pragma unroll
    for (int w = 0; w < 16; ++w) L0.store_one(p, lds, lds + 2 * TILE, w);
    __syncthreads();
    read(fa[0], fb[0], lds, lds + 2 * TILE, 0);
    auto step = [&](int kt, Ld& Lnext, Ld& Lfree) {
      const uint16_t* As = lds + (kt & 1) * TILE;
      const uint16_t* Bs = lds + (2 + (kt & 1)) * TILE;
      uint16_t* Asn = lds + ((kt + 1) & 1) * TILE;
      uint16_t* Bsn = lds + (2 + ((kt + 1) & 1)) * TILE;
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        if (s == S::kLoadStep) Lfree.load(p, m0, n0, int64_t(kt + 2) * BK);
        read(fa[(s + 1) & 1], fb[(s + 1) & 1], As, Bs, s + 1);
        mfmas(fa[s & 1], fb[s & 1]);
        const int w0 = s == 0 ? 0 : s == 1 ? 6 : 11, w1 = s == 0 ? 6 : s == 1 ? 11 : 16;
#pragma unroll
        for (int w = w0; w < w1; ++w) Lnext.store_one(p, Asn, Bsn, kOrder[w]);
        if (s == S::kLoadStep) interleave_kstep<S, true, true>();
        else interleave_kstep<S, false, true>();
        __builtin_amdgcn_sched_barrier(0);
      }
      last_kstep(Asn, Bsn);
    };
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
      step(kt, L1, L0);
      step(kt + 1, L0, L1);
    }
    if (kt < nk) step(kt, L1, L0);
  } else if constexpr (S::kPipe == kPipeOneSet) {
    Ld L;
    L.load(p, m0, n0, 0);
#pragma unroll
    for (int w = 0; w < 16; ++w) L.store_one(p, lds, lds + 2 * TILE, w);
    L.load(p, m0, n0, BK);
    __syncthreads();
    read(fa[0], fb[0], lds, lds + 2 * TILE, 0);
    for (int kt = 0; kt < nk; ++kt) {
      const uint16_t* As = lds + (kt & 1) * TILE;
      const uint16_t* Bs = lds + (2 + (kt & 1)) * TILE;
      uint16_t* Asn = lds + ((kt + 1) & 1) * TILE;
      uint16_t* Bsn = lds + (2 + ((kt + 1) & 1)) * TILE;
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        read(fa[(s + 1) & 1], fb[(s + 1) & 1], As, Bs, s + 1);
        mfmas(fa[s & 1], fb[s & 1]);
        if (s == 0) {
#pragma unroll
          for (int w = 0; w < 16; ++w) L.store_one(p, Asn, Bsn, kOrder[w]);
          interleave_kstep<S, false, true>();
        } else if (s == 1) {
          L.load(p, m0, n0, int64_t(kt + 2) * BK);
          interleave_kstep<S, true, false>();
        } else {
          interleave_kstep<S, false, false>();
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      last_kstep(Asn, Bsn);
    }
  } else {
    Ld L0, L1;
    L0.load(p, m0, n0, 0);
    L1.load(p, m0, n0, BK);
#pragma unroll
    for (int w = 0; w < 16; ++w) L0.store_one(p, lds, lds + 2 * TILE, w);
    __syncthreads();
    auto step = [&](int kt, Ld& Lnext, Ld& Lfree) {
      const uint16_t* As = lds + (kt & 1) * TILE;
      const uint16_t* Bs = lds + (2 + (kt & 1)) * TILE;
      const int nx = (kt + 1) & 1;
      Lfree.load(p, m0, n0, int64_t(kt + 2) * BK);
      read(fa[0], fb[0], As, Bs, 0);
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        if (s < 3) read(fa[(s + 1) & 1], fb[(s + 1) & 1], As, Bs, s + 1);
        mfmas(fa[s & 1], fb[s & 1]);
      }
#pragma unroll
      for (int w = 0; w < 16; ++w) Lnext.store_one(p, lds + nx * TILE, lds + (2 + nx) * TILE, w);
      interleave_tile();
      __syncthreads();
    };
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
      step(kt, L1, L0);
      step(kt + 1, L0, L1);
    }
    if (kt < nk) step(kt, L1, L0);
  }

  // acc[i][j][4g + e] = C[m0 + wm + 32 i + lane % 32][n0 + wn + 32 j + 8 g + 4 (lane / 32) + e]
  if constexpr (V == kFwd || V == kDx) {
    uint16_t* out = static_cast<uint16_t*>(p.out);
    const int64_t row_l = m0 + wm + (lane & 31);
    const int64_t col_l = n0 + wn + 4 * (lane >> 5);
    f32x4 cs[4][4];  // per-channel forward scales of the lane's columns
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t c = col_l + 32 * j + 8 * g;
#pragma unroll
        for (int e = 0; e < 4; ++e) cs[j][g][e] = (V == kFwd && !GRP && c + e < p.N) ? p.s[c + e] : 1.f;
      }
    if ((p.ldo & 7) == 0 && (p.N & 7) == 0 && (reinterpret_cast<uintptr_t>(out) & 15) == 0) {
      // The tile goes through LDS (bf16 [256][256], 16-byte chunks permuted by
      // row as in g_off) and back to memory as whole 512-byte row segments: a
      // store instruction then covers two rows instead of 16 bytes of 32 rows,
      // which shortens the burst of output writes that ends the kernel.
      __syncthreads();  // every wave has read its last fragments
      uint16_t* Cs = lds;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int lr = wm + 32 * i + (lane & 31);
        const float rs = (V == kFwd && ACT && m0 + lr < p.M) ? p.sx[m0 + lr] : 1.f;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            float val[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) val[e] = acc[i][j][4 * g + e] * cs[j][g][e] * rs;
            *reinterpret_cast<u32x2*>(Cs + g_off(lr, wn + 32 * j + 8 * g + 4 * (lane >> 5))) =
                u32x2{pack_bf16x2(val[0], val[1]), pack_bf16x2(val[2], val[3])};
          }
      }
      __syncthreads();
      // thread t writes 16-byte chunk t % 32 of rows 8 ps + t / 32
      const int ch = threadIdx.x & 31;
      const int64_t col = n0 + 8 * ch;
      if (col < p.N) {
#pragma unroll 8
        for (int ps = 0; ps < 32; ++ps) {
          const int lr = 8 * ps + (threadIdx.x >> 5);
          const u32x4 v = *reinterpret_cast<const u32x4*>(Cs + g_off(lr, 8 * ch));
          if (m0 + lr < p.M) *reinterpret_cast<u32x4*>(out + (m0 + lr) * p.ldo + col) = v;
        }
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t row = row_l + 32 * i;
      const float rs = (V == kFwd && ACT && row < p.M) ? p.sx[row] : 1.f;
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int64_t c = col_l + 32 * j + 8 * g;
          float val[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) val[e] = acc[i][j][4 * g + e] * cs[j][g][e] * rs;
          if (row < p.M) {
            uint16_t* dst = out + row * p.ldo + c;
            if (c + 4 <= p.N && (p.ldo & 3) == 0) {
              *reinterpret_cast<u32x2*>(dst) = u32x2{pack_bf16x2(val[0], val[1]), pack_bf16x2(val[2], val[3])};
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (c + e < p.N) dst[e] = __builtin_bit_cast(uint16_t, (__bf16)val[e]);
            }
          }
        }
    }
  } else {
    // ---- dW epilogue: G = s * M * dW staged in LDS as bf16 [row][col], then both
    // rank-r products from LDS; the accumulators are dead once G is staged.
    // The lane holds rows R_i = m0 + wm + 32 i + lane % 32 and, in chunk j (32
    // columns from n0 + wn + 32 j), the columns 8 g + 4 h + e (h = lane / 32).
    const int r = p.r;
    const int nrb = (r + 31) / 32;
    const int half = lane >> 5;
    const int lrow = wm + (lane & 31);  // local row of i = 0
    uint16_t* Gs = lds;

    // columns of chunk j inside N, as a 32-bit mask over the chunk
    uint32_t colok[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t left = p.N - (n0 + wn + 32 * j);
      colok[j] = left >= 32 ? 0xFFFFFFFFu : left <= 0 ? 0u : (1u << left) - 1u;
    }
    // clip-mask bits of chunk j of row R_i: two adjacent 16-bit words, one 4-byte load (rows >= M read 0)
    uint32_t mw[4][4];
    {
      const auto rm = rsrc(p.mask + (m0 + wm) * p.ldm, (p.M - m0 - wm) * p.ldm * 2);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int64_t word = (((lane & 31) + 32 * i) * p.ldm + ((n0 + wn + 32 * j) >> 4)) * 2;
          mw[i][j] = ld32(rm, uint32_t(word)) & colok[j];
        }
    }
    // scales: per channel through LDS, group-wise per (row, chunk) (groups hold whole chunks)
    const auto rsg = rsrc(p.s + m0 * p.ngroups, (p.M - m0) * p.ngroups * 4);  // rows >= M read 0
    if constexpr (!GRP) {
      s_tile[threadIdx.x] = ldf(rsg, uint32_t(threadIdx.x * 4));
      __syncthreads();
    }
    float sc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if constexpr (GRP)
          sc[i][j] = ldf(rsg, uint32_t(((lrow + 32 * i) * p.ngroups + (n0 + wn + 32 * j) / p.gsize) * 4));
        else
          sc[i][j] = s_tile[lrow + 32 * i];
      }

    // scale-gradient partials: ds_part[R_i][chunk] = sum over the chunk of dW (q - z); the lane
    // sums its 16 columns, the lane 32 apart the other 16
    if (p.ds_part) {
      const auto rq = rsrc(p.qd + (m0 + wm) * p.ldqd, (p.M - m0 - wm) * p.ldqd);  // rows >= M read 0
      // without a zero offset the resource is empty and every z reads 0
      const auto rz = p.z ? rsrc(p.z + (m0 + wm) * p.ngroups, (p.M - m0 - wm) * p.ngroups * 4) : rsrc(p.ds_part, 0);
      const auto rd = rsrc(p.ds_part + (m0 + wm) * p.ldds, (p.M - m0 - wm) * p.ldds * 4);
      const bool q8 = p.qd8 != 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rl = (lane & 31) + 32 * i;  // row relative to m0 + wm
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int64_t c0 = n0 + wn + 32 * j;
          const int zi = ld_z(rz, int64_t(rl) * p.ngroups + (GRP ? c0 / p.gsize : 0));
          float sum = 0.f;
          if (q8) {
            // bytes c0 .. c0 + 31 of the row; column 8 g + 4 h + e is byte e of word 2 g + h
            const u32x4 qa = ld128(rq, uint32_t(rl * p.ldqd + c0)), qb = ld128(rq, uint32_t(rl * p.ldqd + c0 + 16));
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const uint32_t w = (2 * g + half) < 4 ? qa[(2 * g + half) & 3] : qb[(2 * g + half) & 3];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const bool ok = (colok[j] >> (8 * g + 4 * half + e)) & 1u;
                sum = __builtin_fmaf(ok ? acc[i][j][4 * g + e] : 0.f, float(sbyte(w, e) - zi), sum);
              }
            }
          } else {
            // nibbles c0 .. c0 + 31 of the row: column 8 g + 4 h + e is nibble 4 h + e of word g
            const u32x4 qv = ld128(rq, uint32_t(rl * p.ldqd + (c0 >> 1)));
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const bool ok = (colok[j] >> (8 * g + 4 * half + e)) & 1u;
                sum = __builtin_fmaf(ok ? acc[i][j][4 * g + e] : 0.f, float(nibble(qv[g], 4 * half + e) - zi), sum);
              }
          }
          sum += __shfl_xor(sum, 32);
          if (half == 0 && colok[j])
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(sum), rd,
                                                  int(uint32_t((rl * p.ldds + (c0 >> 5)) * 4)), 0, 0);
        }
      }
    }

    // G staged as Gs[row][col]: the lane's 4 consecutive columns are one 8-byte write
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int lr = lrow + 32 * i;
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const uint32_t bits = mw[i][j] >> (8 * g + 4 * half);
          float gv[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) gv[e] = (bits >> e) & 1u ? acc[i][j][4 * g + e] * sc[i][j] : 0.f;
          *reinterpret_cast<u32x2*>(Gs + g_off(lr, wn + 32 * j + 8 * g + 4 * half)) =
              u32x2{pack_bf16x2(gv[0], gv[1]), pack_bf16x2(gv[2], gv[3])};
        }
    }

    // stage rank block rb of A (transposed) or B as bf16 [32][256] in `rt_tile`
    auto stage = [&](const float* __restrict__ src, bool is_a, int rb) {
      // unconditional buffer loads, all in flight at once: rows of A past M and ranks of B past r
      // lie outside the resource and read 0; ranks of A past r and columns of B past N are zeroed
      const auto rs = is_a ? rsrc(src + m0 * r, (p.M - m0) * int64_t(r) * 4) : rsrc(src + n0, (int64_t(r) * p.N - n0) * 4);
      if (is_a && (r & 3) == 0) {
        // thread t takes row m0 + t: its 32 ranks as eight 16-byte loads, written transposed
        const int c = threadIdx.x;
        float xv[32];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const u32x4 v = ld128(rs, uint32_t((c * r + 32 * rb + 4 * q) * 4));
#pragma unroll
          for (int e = 0; e < 4; ++e) xv[4 * q + e] = __uint_as_float(v[e]);
        }
#pragma unroll
        for (int rl = 0; rl < 32; ++rl)
          rt_tile[g_off(rl, c)] = uint16_t(pack_bf16x2(32 * rb + rl < r ? xv[rl] : 0.f, 0.f) & 0xFFFFu);
        return;
      }
      const int rho_l = threadIdx.x >> 3, c0 = 32 * (threadIdx.x & 7);
      const int rho = 32 * rb + rho_l;
      float xv[32];
      if (!is_a && (p.N & 3) == 0) {
        // B[rho][n0 + c0 .. +31]: eight 16-byte loads
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const u32x4 v = ld128(rs, uint32_t((int64_t(rho) * p.N + c0 + 4 * q) * 4));
#pragma unroll
          for (int e = 0; e < 4; ++e) xv[4 * q + e] = __uint_as_float(v[e]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 32; ++i) {
          const int c = c0 + i;
          xv[i] = ldf(rs, is_a ? uint32_t((c * r + rho) * 4) : uint32_t((int64_t(rho) * p.N + c) * 4));
        }
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int c = c0 + 8 * q + e;
          x[e] = (rho < r && (is_a || n0 + c < p.N)) ? xv[8 * q + e] : 0.f;  // A[m0 + c][rho] or B[rho][n0 + c]
        }
        u32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = pack_bf16x2(x[2 * e], x[2 * e + 1]);
        *reinterpret_cast<u32x4*>(&rt_tile[g_off(rho_l, c0 + 8 * q)]) = o;
      }
    };

    // dB partial [tm][rho][n0 + j] = sum_i A[m0 + i][rho] G[i][j]; dA partial [tn][m0 + i][rho] = sum_j G[i][j] B[rho][n0 + j]
    const auto rdb = rsrc(p.dB_part + tm * r * p.N + n0, (int64_t(r) * p.N - n0) * 4);
    const auto rda = rsrc(p.dA_part + (tn * p.M + m0) * r, (p.M - m0) * int64_t(r) * 4);
    for (int rb = 0; rb < nrb; ++rb) {
      const int rho = 32 * rb + (lane & 31);
      __syncthreads();  // G staged / previous rank block consumed
      stage(p.Am, true, rb);
      __syncthreads();
      // dB: A operand = A^T rows (rt_tile), B operand = 8 consecutive rows of a G column (LDS transpose loads)
#pragma unroll
      for (int cb2 = 0; cb2 < 2; ++cb2) {
        const int cb = 2 * wave + cb2;            // column block of 32
        const int lj = 32 * cb + (lane & 31);
        f32x16 d;
#pragma unroll
        for (int v = 0; v < 16; ++v) d[v] = 0.f;
#pragma unroll 4
        for (int s2 = 0; s2 < 16; ++s2) {
          const u32x4 aa = *reinterpret_cast<const u32x4*>(&rt_tile[g_off(lane & 31, 16 * s2 + 8 * half)]);
          const u32x4 gb = frag_tr_g(Gs, 32 * cb, 16 * s2, lane);  // G[16 s2 + 8 half .. +7][32 cb + l % 32]
          d = mfma32(aa, gb, d);
        }
        if (n0 + lj < p.N) {
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int rr = 32 * rb + acc_row(v, lane);
            if (rr < r)
              __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(d[v]), rdb, int(uint32_t((int64_t(rr) * p.N + lj) * 4)), 0, 0);
          }
        }
      }
      __syncthreads();
      stage(p.Bm, false, rb);
      __syncthreads();
      // dA: A operand = 8 consecutive columns of a G row (one read), B operand = B rows (rt_tile)
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int rowblk = 2 * wave + h2;
        f32x16 d;
#pragma unroll
        for (int v = 0; v < 16; ++v) d[v] = 0.f;
#pragma unroll 4
        for (int s2 = 0; s2 < 16; ++s2) {
          const u32x4 ga = *reinterpret_cast<const u32x4*>(Gs + g_off(32 * rowblk + (lane & 31), 16 * s2 + 8 * half));
          const u32x4 bb = *reinterpret_cast<const u32x4*>(&rt_tile[g_off(lane & 31, 16 * s2 + 8 * half)]);
          d = mfma32(ga, bb, d);
        }
        if (rho < r) {
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int row = 32 * rowblk + acc_row(v, lane);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(d[v]), rda, int(uint32_t((row * r + rho) * 4)), 0, 0);
          }
        }
      }
    }
  }
}

// Launch one instantiation (all variants share this helper).
template <int V, bool ACT, bool GRP, int OPT>
hipError_t launch_variant(const GemmArgs& p, hipStream_t st) {
  const int64_t ntm = (p.M + BM - 1) / BM, ntn = (p.N + BN - 1) / BN;
  // fast path: 16-byte row vectors (leading dimensions multiples of 8
  // elements) and, for K-contiguous operands, no partial last K-tile
  const bool vec = (p.lda % 8 == 0) && (V != kDw || p.ldb % 8 == 0) && (V == kDw || p.K % BK == 0);
  if (vec) k_gemm<V, ACT, GRP, true, OPT><<<unsigned(ntm * ntn), 256, 0, st>>>(p);
  else k_gemm<V, ACT, GRP, false, OPT><<<unsigned(ntm * ntn), 256, 0, st>>>(p);
  return hipGetLastError();
}

// Run-time choice of the grouped-scale and zero-offset instantiations of one
// family (OPT_BASE: 0 or kOptQ8).
template <int V, bool ACT, int OPT_BASE>
hipError_t launch_zg(bool grouped, bool zp, const GemmArgs& p, hipStream_t st) {
  if (zp) return grouped ? launch_variant<V, ACT, true, OPT_BASE | kOptZ>(p, st) : launch_variant<V, ACT, false, OPT_BASE | kOptZ>(p, st);
  return grouped ? launch_variant<V, ACT, true, OPT_BASE>(p, st) : launch_variant<V, ACT, false, OPT_BASE>(p, st);
}

}  // namespace lrqat
