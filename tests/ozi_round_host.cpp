// Host build of the scheme-I final reduction of the HIP library
// (ozi_round.hpp), for tests/test_ozi_round_host.py.
// stdin: lines "nh e2 H_0 ... H_{nh-1}" (signed 64-bit partial sums).
// stdout per line: the result's bits as 16 hex digits.
#include <cstdio>

#define OZFP4_HD inline
#include "ozi_round.hpp"

using namespace ozfp4;

int main() {
  int nh, e2;
  while (std::scanf("%d %d", &nh, &e2) == 2) {
    if (nh < 1 || nh > kOziMaxGroups) return 2;
    int64_t H[kOziMaxGroups] = {};
    for (int h = 0; h < nh; ++h) {
      long long v;
      if (std::scanf("%lld", &v) != 1) return 2;
      H[h] = (int64_t)v;
    }
    std::printf("%016llx\n", (unsigned long long)bits_of(ozi_compose_round(H, nh, e2)));
  }
  return 0;
}
