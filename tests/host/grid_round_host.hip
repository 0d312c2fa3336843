// Host driver for the library's grid rounding routine: reads lines
// "code f delta_bits_hex" and prints the rounded integer.
#include <cstdio>
#include <cstring>

#include "common.h"

int main() {
  int code, f;
  unsigned bits;
  while (std::scanf("%d %d %x", &code, &f, &bits) == 3) {
    float delta;
    std::memcpy(&delta, &bits, 4);
    std::printf("%d\n", lrqat::grid_round(code, f, delta));
  }
  return 0;
}
