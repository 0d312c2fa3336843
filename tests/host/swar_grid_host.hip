// Host driver for the byte-parallel grid routine: reads lines
// "w incb f b" (w, incb in hex) and prints "q clip" in hex.
#include <cstdio>

#include "grid_swar.h"

int main() {
  unsigned w, incb;
  int f, b;
  while (std::scanf("%x %x %d %d", &w, &incb, &f, &b) == 4) {
    uint32_t clip = 0;
    const uint32_t q = lrqat::swar_grid_q8(w, incb, f, b, clip);
    std::printf("%x %x\n", q, clip);
  }
  return 0;
}
