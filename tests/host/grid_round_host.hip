// Host driver for the library's grid rounding routines: reads lines
// "code f delta_bits_hex" (delta as float32 bits) and prints the float32 and
// the float64 decision.
#include <cstdio>
#include <cstring>

#include "common.h"

int main() {
  int code, f;
  unsigned bits;
  while (std::scanf("%d %d %x", &code, &f, &bits) == 3) {
    float delta;
    std::memcpy(&delta, &bits, 4);
    std::printf("%d %d\n", lrqat::grid_round(code, f, delta), lrqat::grid_round_f64(code, f, double(delta)));
  }
  return 0;
}
