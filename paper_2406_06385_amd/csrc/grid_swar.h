// Byte-parallel integer-grid decision shared by the grid pass and its host test.
#pragma once

#include "common.h"

namespace lrqat {

// Byte-parallel grid of four Q8 codes (one per byte of w) in the regime where
// delta is smaller than the distance of every non-tie code to its rounding
// point (|delta| < 2^-f) and its sign is certain: with n = floor(code / 2^f)
// and cf the f fraction bits, round-half-even(n + cf 2^-f + delta) is n plus
// the carry out of cf + (2^(f-1) - 1) + [delta > 0], since only a tie
// (cf = 2^(f-1)) depends on delta.  incb holds [delta > 0] per byte.  Returns
// the codes as two's complement, in the low nibble of each byte for b <= 4 and
// as whole signed bytes for b >= 5; clip marks (bit 7 of a byte) the codes
// that would leave the grid (n = hi with a carry).
__host__ __device__ __forceinline__ uint32_t swar_grid_q8(uint32_t w, uint32_t incb, int f, int b, uint32_t& clip) {
  const uint32_t ones = 0x01010101u;
  const uint32_t t = (w & (ones * ((1u << f) - 1))) + ones * ((1u << (f - 1)) - 1) + incb;
  const uint32_t carry = (t >> f) & ones;
  const uint32_t mn = ones * ((1u << b) - 1);
  const uint32_t nu = (w >> f) & mn;                       // n as a b-bit pattern per byte
  const uint32_t e = nu ^ (ones * ((1u << (b - 1)) - 1));   // zero where n = hi
  clip |= ~(((e + 0x7F7F7F7Fu) | e) & 0x80808080u) & (carry << 7);
  uint32_t qu = (nu + carry) & mn;
  if (b < 4) qu |= (qu & (ones << (b - 1))) * ((16u - (1u << b)) >> (b - 1));        // sign-extend to 4 bits
  else if (b > 4) qu |= (qu & (ones << (b - 1))) * ((256u - (1u << b)) >> (b - 1));  // to 8 bits
  return qu;
}

}  // namespace lrqat
