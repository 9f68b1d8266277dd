// Single rounding of the exact CRT result to binary32 for the FP32
// emulation: RN_even(x 2^e2) computed from the exact integer, never through
// an FP64 intermediate (rounding twice can move a result by one unit).
// Builtins only, so the host build of a test can check it against exact
// rational arithmetic.
#pragma once

#include "crt_round.hpp"

namespace ozfp4 {

// RN_even(M * 2^e2) to binary32 for the 192-bit magnitude M, with sign:
// quantum 2^(E - 23) for the leading exponent E of the result, at least
// 2^-149 (subnormals); E > 127 or a round-up to 2^128 gives +-inf.
OZFP4_HD float round_scaled_f32(uint64_t w0, uint64_t w1, uint64_t w2, int e2, bool neg) {
  if ((w0 | w1 | w2) == 0) return 0.0f;
  const int n = w2 ? 192 - __builtin_clzll((unsigned long long)w2)
                   : (w1 ? 128 - __builtin_clzll((unsigned long long)w1)
                         : 64 - __builtin_clzll((unsigned long long)w0));
  const int E = n - 1 + e2;
  float r;
  if (E > 127) {
    r = __builtin_huge_valf();
  } else {
    const int qe = (E - 23 > -149 ? E - 23 : -149);
    const int sh = qe - e2;
    if (sh <= 0) {
      r = __builtin_ldexpf((float)w0, e2);  // M < 2^24: exact
    } else {
      uint64_t Rm = shr3(w0, w1, w2, sh);
      const int rb = bit3(w0, w1, w2, sh - 1);
      const bool st = below3(w0, w1, w2, sh - 1);
      if (rb && (st || (Rm & 1ull))) ++Rm;
      r = __builtin_ldexpf((float)Rm, qe);  // Rm <= 2^24: exact or +inf
    }
  }
  return neg ? -r : r;
}

// RN32(x 2^e2) of the exact symmetric CRT result x.
OZFP4_HD float crt_exact_f32(double s0, double s1, double s2, double s3, double q,
                             const CrtConst* __restrict__ cc, int e2) {
  uint64_t w0, w1, w2;
  const bool neg = crt_symmetric(s0, s1, s2, s3, q, cc, &w0, &w1, &w2);
  return round_scaled_f32(w0, w1, w2, e2, neg);
}

}  // namespace ozfp4
