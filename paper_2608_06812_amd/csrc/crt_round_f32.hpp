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

// Fast path for three chunks, in FP64 only: x' (the chunk differences
// after carry normalisation, x' = t 2^84 + d1 2^42 + d0 as in crt_fast3) is
// rounded to odd at 53 bits, and that double, scaled by 2^e2 (exact), is
// converted once to binary32 with round-to-nearest-even. Rounding to odd
// with at least two more bits than the target and then to nearest gives
// the correctly rounded result (Boldo and Melquiond), subnormal binary32
// results included (they have fewer bits still).
//   |t| <= 2: V = (t 2^42 + d1) 2^42 is exact, and Fast2Sum of V and d0
//     (|V| >= 2^42 > d0 unless V = 0) gives x' = hi + lo exactly.
//   |t| >= 3: y = d1 2^42 + d0 is first rounded to odd at 53 bits (a grid
//     of at most 2^31, strictly finer than x''s grid of at least 2^33, so
//     rounding the sum to odd again equals rounding x' to odd), then
//     Fast2Sum of t 2^84 and that value gives hi + lo.
// Round to odd of hi + lo: hi if lo = 0, else the neighbour of x' whose
// last significand bit is 1 (hi itself if odd, else one unit towards lo).
// Gives up, like crt_fast3, when |x'| may lie outside (-P/2, P/2] or when
// x' 2^e2 may fall below the FP64 normal range.
OZFP4_HD bool crt_fast3_f32(double s0, double s1, double s2, double q,
                            const CrtConst* __restrict__ cc, int e2, float* out) {
  constexpr double kC = 0x1p42, kCi = 0x1p-42;
  const double v0 = __builtin_fma(-q, cc->Pc[0], s0);
  double v1 = __builtin_fma(-q, cc->Pc[1], s1);
  const double v2 = __builtin_fma(-q, cc->Pc[2], s2);
  const double c0 = __builtin_floor(v0 * kCi);
  const double d0 = __builtin_fma(-c0, kC, v0);
  v1 += c0;
  const double c1 = __builtin_floor(v1 * kCi);
  const double d1 = __builtin_fma(-c1, kC, v1);
  const double t = v2 + c1;
  double a, b;   // x' (or x' with y rounded to odd) = a + b, |a| >= |b| or a = 0
  if (__builtin_fabs(t) <= 2.0) {
    a = __builtin_fma(t, kC, d1) * kC;
    b = d0;
  } else {
    const double D1 = d1 * kC;
    const double sy = D1 + d0;
    const double ey = d0 - (sy - D1);
    uint64_t yb = bits_of(sy);
    yb = ey > 0.0 ? (yb | 1ull) : ((ey < 0.0 && !(yb & 1ull)) ? yb - 1ull : yb);
    a = t * 0x1p84;
    b = double_of(yb);
  }
  const double hi = a + b;
  const double lo = b - (hi - a);
  uint64_t hb = bits_of(hi);
  if (lo != 0.0) {
    if ((lo > 0.0) == (hi > 0.0)) hb |= 1ull;   // |x'| above |hi|
    else if (!(hb & 1ull)) hb -= 1ull;          // |x'| below |hi|
  }
  const double r = double_of(hb);
  if (!(__builtin_fabs(r) < cc->sym_limit)) return false;
  if (r != 0.0) {
    int fe;
    (void)__builtin_frexp(r, &fe);
    if (fe + e2 <= -1020) return false;
  }
  *out = (float)__builtin_ldexp(r, e2);
  return true;
}

}  // namespace ozfp4
