// Host build of the two-term split's final step (crt_split.hpp), for
// tests/test_crt_split_host.py.
// stdin: lines "d e2  s11 a11 b11 c11  s12 a12 b12 c12  s22 a22 b22 c22"
//   (for each product: sign 0/1 and the three 64-bit words of the
//   magnitude, low first, in hex);
// stdout per line: the FP64 result bits of RN((X11 2^2d + X12 2^d + X22) 2^e2)
// in 16 hex digits.
#include <cstdio>
#include <cstdint>

#define OZFP4_HD inline
#include "crt_split.hpp"

using namespace ozfp4;

int main() {
  int d, e2;
  while (std::scanf("%d %d", &d, &e2) == 2) {
    uint64_t acc[4] = {0, 0, 0, 0};
    const int shifts[3] = {2 * d, d, 0};
    for (int p = 0; p < 3; ++p) {
      int sg;
      unsigned long long a, b, c;
      if (std::scanf("%d %llx %llx %llx", &sg, &a, &b, &c) != 4) return 2;
      add_shifted256(acc, a, b, c, sg != 0, shifts[p]);
    }
    const double r = round_scaled256(acc, e2);
    uint64_t bits;
    __builtin_memcpy(&bits, &r, 8);
    std::printf("%016llx\n", (unsigned long long)bits);
  }
  return 0;
}
