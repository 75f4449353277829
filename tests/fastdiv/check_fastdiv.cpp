// Host check of the kernels' division by a launch-fixed divisor (make_fastdiv
// and fdiv in csrc/common.h): the quotient equals n / d for small, large
// and random dividends in [0, 2^31) over divisors from 1 to 2^31 - 1,
// including powers of two and their neighbours.  Exits 1 on any mismatch.
#include <cstdio>
#include <cstdint>
#include "common.h"
using namespace cnnlib;
int main() {
  uint64_t bad = 0, n_checked = 0;
  uint32_t ds[] = {1, 2, 3, 5, 7, 9, 28, 30, 55, 56, 58, 112, 229, 784, 3025, 12544, 52441,
                   65535, 65536, 65537, 1000003, 1u << 20, (1u << 20) + 1, 0x3fffffffu, 0x40000000u,
                   0x40000001u, 0x7ffffffeu, 0x7fffffffu};
  uint32_t seed = 12345;
  for (uint32_t d : ds) {
    const FastDiv f = make_fastdiv(d);
    for (int i = 0; i < 200000; ++i) {
      seed = seed * 1664525u + 1013904223u;
      uint32_t n = i < 64 ? (uint32_t)i : i < 128 ? 0x7fffffffu - (uint32_t)(i - 64) : (seed & 0x7fffffffu);
      if (i >= 128 && (i & 3) == 0) n = (uint32_t)((uint64_t)(seed >> 8) % 64 + (uint64_t)d * ((seed & 0xffff) % (0x7fffffffu / d + 1)));
      if (n > 0x7fffffffu) continue;
      ++n_checked;
      if ((uint32_t)fdiv((int)n, f) != n / d) ++bad;
    }
  }
  printf("checked %llu bad %llu\n", (unsigned long long)n_checked, (unsigned long long)bad);
  return bad != 0;
}
