// Device-side building blocks shared by the LR-QAT kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace lrqat {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// ---------------------------------------------------------------- conversions

// Two floats -> packed bfloat16 pair (round to nearest even; v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2 v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// Signed 4-bit field `idx` (0..7) of a 32-bit word.
__device__ __forceinline__ int nibble(uint32_t w, int idx) {
  return int(w << (28 - 4 * idx)) >> 28;
}
// Signed byte `idx` (0..3) of a 32-bit word.
__device__ __forceinline__ int sbyte(uint32_t w, int idx) {
  return int(w << (24 - 8 * idx)) >> 24;
}

// v_perm_b32 helpers: low (resp. high) 16-bit halves of two words -> one word
// {a.half, b.half} with a in the low half.
__device__ __forceinline__ uint32_t perm_lo16(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x05040100u);
}
__device__ __forceinline__ uint32_t perm_hi16(uint32_t a, uint32_t b) {
  return __builtin_amdgcn_perm(b, a, 0x07060302u);
}

// ---------------------------------------------------------------- MFMA

// D(32x32, f32) += A(32x16, bf16) * B(16x32, bf16).  Lane l supplies row l%32
// of A and column l%32 of B, each with the 8 K-values of K-half l/32.  The
// accumulator element v of lane l is D[8*(v/4) + 4*(l/32) + v%4][l%32].
__device__ __forceinline__ f32x16 mfma32(const u32x4& a, const u32x4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ int acc_row(int v, int lane) { return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3); }

// ---------------------------------------------------------------- the grid decision
// round-half-even(u) for u = code * 2^-f + delta, taken without absorbing a
// small delta into the stored value.  With n = floor(code / 2^f) and the
// fraction bits cf = code mod 2^f,
//     u = n + 1/2 + w,   w = (cf * 2^-f - 1/2) + delta,
// where the bracket is exact in float32.  For non-integer w the nearest
// integer is n + ceil(w); an integer w is a tie between n + w and n + w + 1,
// resolved to the even one.  float32 keeps the sign of w exact (it is 0 only
// when the bracket cancels delta exactly), so near the usual decision point
// w = 0 the only error is that of delta itself.  f = 0 is integer Phi0.
__host__ __device__ __forceinline__ int grid_round(int code, int f, float delta, float* margin = nullptr) {
  const int n = code >> f;
  const int cf = code & ((1 << f) - 1);
  const float w = (float(cf) * __builtin_bit_cast(float, uint32_t(127 - f) << 23) - 0.5f) + delta;
  const float cw = __builtin_ceilf(w);
  int ut = n + int(cw);
  if (cw == w) ut += ut & 1;
  if (margin) {
    // distance to the nearest decision point nd, less the rounding error of the
    // float32 sum there (at most 2^-23 |nd|; the sum is exact near nd = 0)
    const float nd = __builtin_rintf(w);
    *margin = __builtin_fabsf(w - nd) - 0x1p-23f * __builtin_fabsf(nd);
  }
  return ut;
}

// The same decision with delta in float64, for elements whose float32 margin
// does not exceed the error bound of the float32 delta.
__host__ __device__ __forceinline__ int grid_round_f64(int code, int f, double delta) {
  const int n = code >> f;
  const int cf = code & ((1 << f) - 1);
  const double w = (double(cf) * __builtin_bit_cast(double, uint64_t(1023 - f) << 52) - 0.5) + delta;
  const double cw = __builtin_ceil(w);
  int ut = n + int(cw);
  if (cw == w) ut += ut & 1;
  return ut;
}

}  // namespace lrqat
