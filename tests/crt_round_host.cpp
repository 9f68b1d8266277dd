// Host build of the CRT reconstruction and rounding functions of the HIP
// library (crt_round.hpp), for tests/test_crt_round_host.py.
// stdin: lines "L e2 r_0 ... r_{L-1}" (residues in [0, m_l)).
// stdout per line: "<fast-or-exact result bits> <exact-path bits> <1 if the
// fast path decided> <binary32 result bits>", 16, 16 and 8 hex digits.
#include <cstdio>
#include <cstring>
#include <vector>

#define OZFP4_HD inline
#include "crt_round.hpp"
#include "crt_round_f32.hpp"

using namespace ozfp4;

int main() {
  static HostTables T;
  if (!build_tables(T)) {
    std::printf("tables failed\n");
    return 1;
  }
  int L, e2;
  while (std::scanf("%d %d", &L, &e2) == 2) {
    if (L < 2 || L > kMaxModuli) return 2;
    std::vector<int> r(L);
    for (int l = 0; l < L; ++l)
      if (std::scanf("%d", &r[l]) != 1) return 2;
    const CrtConst* cc = &T.crt[L];
    const int NC = cc->nc;
    double sig[4] = {0, 0, 0, 0};
    for (int l = 0; l < L; ++l)
      for (int c = 0; c < NC; ++c) sig[c] = __builtin_fma((double)r[l], cc->W[l][c], sig[c]);
    double Qe = sig[NC - 1] * cc->Qc[NC - 1];
    for (int c = NC - 2; c >= 0; --c) Qe = __builtin_fma(sig[c], cc->Qc[c], Qe);
    const double q = __builtin_rint(Qe);
    double out = 0.0;
    bool fast = false;
    if (NC == 3) fast = crt_fast3(sig[0], sig[1], sig[2], q, cc, e2, &out);
    const double ex = crt_exact(sig[0], sig[1], sig[2], NC == 4 ? sig[3] : 0.0, q, cc, e2);
    if (!fast) out = ex;
    const float f = crt_exact_f32(sig[0], sig[1], sig[2], NC == 4 ? sig[3] : 0.0, q, cc, e2);
    float ff = f;
    bool fast32 = false;
    if (NC == 3) fast32 = crt_fast3_f32(sig[0], sig[1], sig[2], q, cc, e2, &ff);
    std::printf("%016llx %016llx %d %08x %08x %d\n", (unsigned long long)bits_of(out),
                (unsigned long long)bits_of(ex), fast ? 1 : 0, __builtin_bit_cast(uint32_t, f),
                __builtin_bit_cast(uint32_t, ff), fast32 ? 1 : 0);
  }
  return 0;
}
