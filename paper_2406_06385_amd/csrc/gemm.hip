// bf16 MFMA GEMMs of the LR-QAT layer on gfx950.
//
//   kFwd  Y  = X_hat W_hat^T      M = T, N = m, K = k   (Section 3, Eq. lr_qat)
//   kDx   dX = dY W_hat           M = T, N = k, K = m
//   kDw   dW = dY^T X_hat         M = m, N = k, K = T, never stored: the
//         epilogue forms G = s * M * dW and the rank-r partial products
//         G B^T and A^T G (Section 3, STE gradients w.r.t. A and B).
//
// W_hat enters as the packed integer grid q written by the grid pass; the
// operand loaders unpack it into bfloat16 tiles in LDS (exact for |q| <= 8),
// with the scale s applied in the epilogue (forward, per channel) or folded
// into the tile (dX, and the forward with group-wise scales).
//
// Block tile 256 x 256 x 64, four waves in a 2 x 2 arrangement, each wave a
// 128 x 128 sub-tile of 4 x 4 MFMA 32x32x16 blocks.  Two LDS stages of
// (256 + 256) x 64 bfloat16 (128 KiB); the next K-tile is fetched into
// registers while the current one feeds the MFMAs.
#include "kernels.h"

namespace lrqat {

constexpr int BM = GEMM_BM, BN = GEMM_BN, BK = GEMM_BK;
constexpr int STAGE = (BM + BN) * BK;  // bfloat16 elements per LDS stage

// ------------------------------------------------------------------ buffer resources
// Operands are read with raw buffer loads.  A load past the resource's
// num_records returns zeros, so a tile that overhangs the end of a tensor
// needs no per-lane branch: each resource starts at the tile's first row.
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

// 8 bfloat16 at element offset `off` of a row (16-bit loads: rows not 16-byte aligned).
__device__ __forceinline__ u32x4 ld8_bf16_scalar(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  u32x4 v;
#pragma unroll
  for (int q = 0; q < 4; ++q) v[q] = ld16(r, 2 * (off + 2 * q)) | (ld16(r, 2 * (off + 2 * q + 1)) << 16);
  return v;
}

// Zero the elements of an 8-wide bfloat16 chunk at column kk that lie at or past K.
__device__ __forceinline__ u32x4 mask_tail(u32x4 v, int64_t kk, int64_t K) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t lo = (kk + 2 * q < K) ? 0x0000FFFFu : 0u, hi = (kk + 2 * q + 1 < K) ? 0xFFFF0000u : 0u;
    v[q] &= lo | hi;
  }
  return v;
}

// ------------------------------------------------------------------ K-contiguous bf16 source
// 256 x 64 tile of a row-major [rows][K] bfloat16 matrix; thread t loads
// chunk t%8 of rows t/8 + 32 i.
struct RegsKc {
  u32x4 v[8];
};

template <bool VEC>
__device__ __forceinline__ void load_kc_bf16(RegsKc& R, const uint16_t* __restrict__ src, int64_t ld,
                                             int64_t row0, int64_t nrows, int64_t k0, int64_t K) {
  const int t = threadIdx.x;
  const auto r = rsrc(src + row0 * ld, (nrows - row0) * ld * 2);
  const int64_t kk = k0 + 8 * (t & 7);
  const bool tail = k0 + GEMM_BK > K;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t off = uint32_t(((t >> 3) + 32 * i) * ld + kk);
    R.v[i] = VEC ? ld128(r, 2 * off) : ld8_bf16_scalar(r, off);
  }
  if (tail) {
#pragma unroll
    for (int i = 0; i < 8; ++i) R.v[i] = mask_tail(R.v[i], kk, K);
  }
}

__device__ __forceinline__ void store_kc(uint16_t* tile, const RegsKc& R) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 8; ++i) *reinterpret_cast<u32x4*>(tile + tile_off((t >> 3) + 32 * i, t & 7)) = R.v[i];
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
  const int64_t kk = k0 + 8 * (t & 7);
#pragma unroll
  for (int i = 0; i < 8; ++i) R.v[i] = ld64(r, uint32_t(((t >> 3) + 32 * i) * ld + kk));
}

__device__ __forceinline__ void store_kc_i8(uint16_t* tile, const RegsKc8& R) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t w = R.v[i][q >> 1];
      o[q] = pack_bf16x2(float(sbyte(w, 2 * (q & 1))), float(sbyte(w, 2 * (q & 1) + 1)));
    }
    *reinterpret_cast<u32x4*>(tile + tile_off((t >> 3) + 32 * i, t & 7)) = o;
  }
}

// ------------------------------------------------------------------ packed q, K-contiguous (forward B)
// 256 weight rows x 64 K-values = 256 x 32 bytes; thread t takes 16 bytes
// (32 values) of rows t/2 and t/2 + 128.  q is zero past column k.
struct RegsQKc {
  u32x4 v[2];
  float sc[2];
};

template <bool GRP>
__device__ __forceinline__ void load_q_kc(RegsQKc& R, const GemmArgs& p, int64_t row0, int64_t k0) {
  const int t = threadIdx.x;
  const int64_t kk = k0 + 32 * (t & 1);
  const auto rq = rsrc(static_cast<const uint8_t*>(p.b) + row0 * p.ldb, (p.N - row0) * p.ldb);
#pragma unroll
  for (int i = 0; i < 2; ++i) R.v[i] = ld128(rq, uint32_t(((t >> 1) + 128 * i) * p.ldb + (kk >> 1)));
  if (GRP) {
    const auto rs = rsrc(p.s + row0 * p.ngroups, (p.N - row0) * p.ngroups * 4);
    const int64_t g = kk / p.gsize;
#pragma unroll
    for (int i = 0; i < 2; ++i) R.sc[i] = ldf(rs, uint32_t((((t >> 1) + 128 * i) * p.ngroups + g) * 4));
  }
}

template <bool GRP>
__device__ __forceinline__ void store_q_kc(uint16_t* tile, const RegsQKc& R) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = (t >> 1) + 128 * i;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint32_t w = R.v[i][c];
      u32x4 o;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float a = float(nibble(w, 2 * q)), b = float(nibble(w, 2 * q + 1));
        if (GRP) {
          a *= R.sc[i];
          b *= R.sc[i];
        }
        o[q] = pack_bf16x2(a, b);
      }
      *reinterpret_cast<u32x4*>(tile + tile_off(row, 4 * (t & 1) + c)) = o;
    }
  }
}

// ------------------------------------------------------------------ packed q, K-strided (dX B)
// K = weight rows (m), N = weight columns (k).  Thread t: 8 columns
// (8 t%32 .. +7 -> 4 bytes) of 8 rows (8 (t/32) .. +7); each value is
// scaled by its row's (or row-group's) s before the bfloat16 rounding.
struct RegsQKs {
  uint32_t w[8];
  float sc[8];
};

template <bool GRP>
__device__ __forceinline__ void load_q_ks(RegsQKs& R, const GemmArgs& p, int64_t n0, int64_t k0) {
  const int t = threadIdx.x;
  const int64_t col = n0 + 8 * (t & 31);
  const int64_t rl = 8 * (t >> 5);
  const auto rq = rsrc(static_cast<const uint8_t*>(p.b) + k0 * p.ldb, (p.K - k0) * p.ldb);
#pragma unroll
  for (int e = 0; e < 8; ++e) R.w[e] = ld32(rq, uint32_t((rl + e) * p.ldb + (col >> 1)));
  if (GRP) {
    const auto rs = rsrc(p.s + k0 * p.ngroups, (p.K - k0) * p.ngroups * 4);
    const int64_t g = col / p.gsize;
#pragma unroll
    for (int e = 0; e < 8; ++e) R.sc[e] = ldf(rs, uint32_t(((rl + e) * p.ngroups + g) * 4));
  } else {
    const auto rs = rsrc(p.s + k0, (p.K - k0) * 4);
#pragma unroll
    for (int e = 0; e < 8; ++e) R.sc[e] = ldf(rs, uint32_t((rl + e) * 4));
  }
}

__device__ __forceinline__ void store_q_ks(uint16_t* tile, const RegsQKs& R) {
  const int t = threadIdx.x;
  const int kg = t >> 5;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      o[q] = pack_bf16x2(float(nibble(R.w[2 * q], c)) * R.sc[2 * q],
                         float(nibble(R.w[2 * q + 1], c)) * R.sc[2 * q + 1]);
    *reinterpret_cast<u32x4*>(tile + tile_off(8 * (t & 31) + c, kg)) = o;
  }
}

// ------------------------------------------------------------------ bf16, K-strided (dW A and B)
// Tile rows = the index contiguous in memory, K = the strided (token) index.
// Thread t: 8 consecutive tile rows (8 t%32 .. +7, one 16-byte vector) of
// 8 K-lines (8 (t/32) .. +7), transposed in registers into 8 chunks.
// Columns past the tensor's width only feed output rows/columns that the
// epilogue discards; K-lines past the end read as zeros.
struct RegsKs {
  u32x4 v[8];
};

template <bool VEC>
__device__ __forceinline__ void load_ks_bf16(RegsKs& R, const uint16_t* __restrict__ src, int64_t ld,
                                             int64_t c0, int64_t k0, int64_t K) {
  const int t = threadIdx.x;
  const int64_t col = c0 + 8 * (t & 31);
  const int64_t rl = 8 * (t >> 5);
  const auto r = rsrc(src + k0 * ld, (K - k0) * ld * 2);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t off = uint32_t((rl + e) * ld + col);
    R.v[e] = VEC ? ld128(r, 2 * off) : ld8_bf16_scalar(r, off);
  }
}

__device__ __forceinline__ void store_ks_bf16(uint16_t* tile, const RegsKs& R) {
  const int t = threadIdx.x;
  const int kg = t >> 5;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t a = R.v[2 * q][c >> 1], b = R.v[2 * q + 1][c >> 1];
      o[q] = (c & 1) ? perm_hi16(a, b) : perm_lo16(a, b);
    }
    *reinterpret_cast<u32x4*>(tile + tile_off(8 * (t & 31) + c, kg)) = o;
  }
}

// int8 codes n [T][ld] times s_x[t], K-strided (dW B under W4A8).
struct RegsKs8 {
  u32x2 v[8];
  float sx[8];
};

__device__ __forceinline__ void load_ks_i8(RegsKs8& R, const int8_t* __restrict__ src, int64_t ld,
                                           const float* __restrict__ sx, int64_t c0, int64_t k0, int64_t K) {
  const int t = threadIdx.x;
  const int64_t col = c0 + 8 * (t & 31);
  const int64_t rl = 8 * (t >> 5);
  const auto r = rsrc(src + k0 * ld, (K - k0) * ld);
  const auto rs = rsrc(sx + k0, (K - k0) * 4);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    R.v[e] = ld64(r, uint32_t((rl + e) * ld + col));
    R.sx[e] = ldf(rs, uint32_t((rl + e) * 4));
  }
}

__device__ __forceinline__ void store_ks_i8(uint16_t* tile, const RegsKs8& R) {
  const int t = threadIdx.x;
  const int kg = t >> 5;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      o[q] = pack_bf16x2(float(sbyte(R.v[2 * q][c >> 2], c & 3)) * R.sx[2 * q],
                         float(sbyte(R.v[2 * q + 1][c >> 2], c & 3)) * R.sx[2 * q + 1]);
    *reinterpret_cast<u32x4*>(tile + tile_off(8 * (t & 31) + c, kg)) = o;
  }
}

// ------------------------------------------------------------------ the kernel

template <int V, bool ACT, bool GRP, bool VEC>
struct Loader;

template <bool ACT, bool GRP, bool VEC>
struct Loader<kFwd, ACT, GRP, VEC> {
  typename std::conditional<ACT, RegsKc8, RegsKc>::type ra;
  RegsQKc rb;
  __device__ __forceinline__ void load(const GemmArgs& p, int64_t m0, int64_t n0, int64_t k0) {
    if constexpr (ACT) load_kc_i8(ra, static_cast<const int8_t*>(p.a), p.lda, m0, p.M, k0);
    else load_kc_bf16<VEC>(ra, static_cast<const uint16_t*>(p.a), p.lda, m0, p.M, k0, p.K);
    load_q_kc<GRP>(rb, p, n0, k0);
  }
  __device__ __forceinline__ void store(uint16_t* As, uint16_t* Bs) {
    if constexpr (ACT) store_kc_i8(As, ra);
    else store_kc(As, ra);
    store_q_kc<GRP>(Bs, rb);
  }
};

template <bool ACT, bool GRP, bool VEC>
struct Loader<kDx, ACT, GRP, VEC> {
  RegsKc ra;
  RegsQKs rb;
  __device__ __forceinline__ void load(const GemmArgs& p, int64_t m0, int64_t n0, int64_t k0) {
    load_kc_bf16<VEC>(ra, static_cast<const uint16_t*>(p.a), p.lda, m0, p.M, k0, p.K);
    load_q_ks<GRP>(rb, p, n0, k0);
  }
  __device__ __forceinline__ void store(uint16_t* As, uint16_t* Bs) {
    store_kc(As, ra);
    store_q_ks(Bs, rb);
  }
};

template <bool ACT, bool GRP, bool VEC>
struct Loader<kDw, ACT, GRP, VEC> {
  RegsKs ra;
  typename std::conditional<ACT, RegsKs8, RegsKs>::type rb;
  __device__ __forceinline__ void load(const GemmArgs& p, int64_t m0, int64_t n0, int64_t k0) {
    load_ks_bf16<VEC>(ra, static_cast<const uint16_t*>(p.a), p.lda, m0, k0, p.K);
    if constexpr (ACT) load_ks_i8(rb, static_cast<const int8_t*>(p.b), p.ldb, p.sx, n0, k0, p.K);
    else load_ks_bf16<VEC>(rb, static_cast<const uint16_t*>(p.b), p.ldb, n0, k0, p.K);
  }
  __device__ __forceinline__ void store(uint16_t* As, uint16_t* Bs) {
    store_ks_bf16(As, ra);
    if constexpr (ACT) store_ks_i8(Bs, rb);
    else store_ks_bf16(Bs, rb);
  }
};

// Offset of G[i][j] in the 256 x 256 bfloat16 staging tile of the dW epilogue
// (16-byte chunks of a 512-byte row permuted by i mod 16).
__device__ __forceinline__ int g_off(int i, int j) { return i * 256 + ((((j >> 3) ^ (i & 15))) << 3) + (j & 7); }

template <int V, bool ACT, bool GRP, bool VEC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_gemm(GemmArgs p) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t ntm = (p.M + BM - 1) / BM;
  const int64_t tm = blockIdx.x % ntm, tn = blockIdx.x / ntm;
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int wm = (wave >> 1) * 128, wn = (wave & 1) * 128;

  f32x16 acc[4][4];
  #pragma unroll
  for (int a = 0; a < 4; ++a)
    #pragma unroll
    for (int b = 0; b < 4; ++b)
      #pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;

  Loader<V, ACT, GRP, VEC> ld;
  const int nk = int((p.K + BK - 1) / BK);
  if (nk > 0) {
    ld.load(p, m0, n0, 0);
    ld.store(lds, lds + BM * BK);
    __syncthreads();
  }
  for (int kt = 0; kt < nk; ++kt) {
    uint16_t* As = lds + (kt & 1) * STAGE;
    uint16_t* Bs = As + BM * BK;
    const bool more = kt + 1 < nk;
    if (more) ld.load(p, m0, n0, int64_t(kt + 1) * BK);
    #pragma unroll
    for (int s = 0; s < 4; ++s) {
      u32x4 af[4], bf[4];
      const int ch = 2 * s + (lane >> 5);
      #pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const u32x4*>(As + tile_off(wm + 32 * i + (lane & 31), ch));
      #pragma unroll
      for (int j = 0; j < 4; ++j) bf[j] = *reinterpret_cast<const u32x4*>(Bs + tile_off(wn + 32 * j + (lane & 31), ch));
      #pragma unroll
      for (int i = 0; i < 4; ++i)
        #pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma32(af[i], bf[j], acc[i][j]);
    }
    if (more) {
      uint16_t* An = lds + ((kt + 1) & 1) * STAGE;
      ld.store(An, An + BM * BK);
    }
    __syncthreads();
  }

  if constexpr (V == kFwd || V == kDx) {
    uint16_t* out = static_cast<uint16_t*>(p.out);
    #pragma unroll
    for (int i = 0; i < 4; ++i)
      #pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t col = n0 + wn + 32 * j + (lane & 31);
        if (col >= p.N) continue;
        float cs = 1.f;
        if (V == kFwd && !GRP) cs = p.s[col];
        #pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int64_t row = m0 + wm + 32 * i + acc_row(v, lane);
          if (row >= p.M) continue;
          float val = acc[i][j][v] * cs;
          if (V == kFwd && ACT) val *= p.sx[row];
          out[row * p.ldo + col] = __builtin_bit_cast(uint16_t, (__bf16)val);
        }
      }
  } else {
    // ---- G = s * M * dW, kept in registers (fp32) and staged in LDS (bf16)
    uint16_t* Gs = lds;
    #pragma unroll
    for (int i = 0; i < 4; ++i)
      #pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int lj = wn + 32 * j + (lane & 31);
        const int64_t col = n0 + lj;
        #pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int li = wm + 32 * i + acc_row(v, lane);
          const int64_t row = m0 + li;
          float g = 0.f;
          if (row < p.M && col < p.N) {
            const float sc = GRP ? p.s[row * p.ngroups + col / p.gsize] : p.s[row];
            const int bit = (p.mask[row * p.ldm + (col >> 3)] >> (col & 7)) & 1;
            g = bit ? acc[i][j][v] * sc : 0.f;
          }
          acc[i][j][v] = g;
          Gs[g_off(li, lj)] = __builtin_bit_cast(uint16_t, (__bf16)g);
        }
      }
    __syncthreads();

    const int r = p.r;
    const int nrb = (r + 31) / 32;
    const int half = lane >> 5;
    // ---- dA partial [tn][row][rho] = sum_j G[row][j] B[rho][n0 + j]   (A operand from LDS)
    for (int pr = wave; pr < 8 * nrb; pr += 4) {
      const int rowblk = pr & 7, rb = pr >> 3;
      const int rho = 32 * rb + (lane & 31);
      f32x16 d;
      #pragma unroll
      for (int v = 0; v < 16; ++v) d[v] = 0.f;
      #pragma unroll
      for (int s = 0; s < 16; ++s) {
        const int li = 32 * rowblk + (lane & 31);
        const u32x4 aop = *reinterpret_cast<const u32x4*>(Gs + g_off(li, 16 * s + 8 * half));
        float x[8];
        const int64_t jb = n0 + 16 * s + 8 * half;
        #pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = (rho < r && jb + e < p.N) ? p.Bm[int64_t(rho) * p.N + jb + e] : 0.f;
        u32x4 bop;
        #pragma unroll
        for (int q = 0; q < 4; ++q) bop[q] = pack_bf16x2(x[2 * q], x[2 * q + 1]);
        d = mfma32(aop, bop, d);
      }
      if (rho < r) {
        #pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int64_t row = m0 + 32 * rowblk + acc_row(v, lane);
          if (row < p.M) p.dA_part[(tn * p.M + row) * r + rho] = d[v];
        }
      }
    }
    // ---- dB partial [2 tm + wave row][rho][col] = sum_i A[m0 + i][rho] G[i][col]  (G from registers)
    const int64_t part = 2 * tm + (wave >> 1);
    for (int rb = 0; rb < nrb; ++rb) {
      const int rho = 32 * rb + (lane & 31);
      u32x4 aop[4][2];
      #pragma unroll
      for (int i = 0; i < 4; ++i)
        #pragma unroll
        for (int s = 0; s < 2; ++s) {
          float x[8];
          #pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int64_t row = m0 + wm + 32 * i + acc_row(8 * s + e, lane);
            x[e] = (rho < r && row < p.M) ? p.Am[row * r + rho] : 0.f;
          }
          #pragma unroll
          for (int q = 0; q < 4; ++q) aop[i][s][q] = pack_bf16x2(x[2 * q], x[2 * q + 1]);
        }
      #pragma unroll
      for (int j = 0; j < 4; ++j) {
        f32x16 d;
        #pragma unroll
        for (int v = 0; v < 16; ++v) d[v] = 0.f;
        #pragma unroll
        for (int i = 0; i < 4; ++i)
          #pragma unroll
          for (int s = 0; s < 2; ++s) {
            u32x4 gop;
            #pragma unroll
            for (int q = 0; q < 4; ++q) gop[q] = pack_bf16x2(acc[i][j][8 * s + 2 * q], acc[i][j][8 * s + 2 * q + 1]);
            d = mfma32(aop[i][s], gop, d);
          }
        const int64_t col = n0 + wn + 32 * j + (lane & 31);
        if (col < p.N) {
          #pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int rr = 32 * rb + acc_row(v, lane);
            if (rr < r) p.dB_part[(part * r + rr) * p.N + col] = d[v];
          }
        }
      }
    }
  }
}

// Deterministic sum of partial buffers: out = (accumulate ? out : 0) + c * sum_p part[p].
__global__ __launch_bounds__(256) void k_reduce(const float* __restrict__ part, int64_t nparts, int64_t n,
                                                float* __restrict__ out, float c, int accumulate) {
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= n) return;
  float s = 0.f;
  for (int64_t q = 0; q < nparts; ++q) s += part[q * n + idx];
  out[idx] = (accumulate ? out[idx] : 0.f) + c * s;
}

template <int V, bool ACT, bool GRP>
static hipError_t launch_variant(const GemmArgs& p, hipStream_t st) {
  const int64_t ntm = (p.M + BM - 1) / BM, ntn = (p.N + BN - 1) / BN;
  // 16-byte row vectors need leading dimensions that are multiples of 8 elements
  const bool vec = (p.lda % 8 == 0) && (V != kDw || p.ldb % 8 == 0);
  if (vec) k_gemm<V, ACT, GRP, true><<<unsigned(ntm * ntn), 256, 0, st>>>(p);
  else k_gemm<V, ACT, GRP, false><<<unsigned(ntm * ntn), 256, 0, st>>>(p);
  return hipGetLastError();
}

hipError_t launch_gemm(GemmVariant v, bool act, bool grouped, const GemmArgs& p, hipStream_t st) {
  switch (v) {
    case kFwd:
      if (act) return grouped ? launch_variant<kFwd, true, true>(p, st) : launch_variant<kFwd, true, false>(p, st);
      return grouped ? launch_variant<kFwd, false, true>(p, st) : launch_variant<kFwd, false, false>(p, st);
    case kDx:
      return grouped ? launch_variant<kDx, false, true>(p, st) : launch_variant<kDx, false, false>(p, st);
    case kDw:
      if (act) return grouped ? launch_variant<kDw, true, true>(p, st) : launch_variant<kDw, true, false>(p, st);
      return grouped ? launch_variant<kDw, false, true>(p, st) : launch_variant<kDw, false, false>(p, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_reduce(const float* part, int64_t nparts, int64_t n, float* out, float c, int accumulate,
                         hipStream_t st) {
  k_reduce<<<unsigned((n + 255) / 256), 256, 0, st>>>(part, nparts, n, out, c, accumulate);
  return hipGetLastError();
}

}  // namespace lrqat
