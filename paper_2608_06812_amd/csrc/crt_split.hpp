// Final step of the two-term split (an extension of Sec. IV-B): the three
// exact symmetric integers of the split products, X11 = A1 B1,
// X12 = A1 B2 + A2 B1 and X22 = A2 B2 (each a sign and a 192-bit magnitude
// from the CRT's exact path, Sec. V-B), are combined into
// X = X11 2^(2d) + X12 2^d + X22 in 256-bit two's complement and X 2^e2 is
// rounded once to FP64. With 53-bit capacities (d <= 53) and k <= 2^16,
// |X11|, |X12| <= k 2^106 and |X22| <= k 2^104, so |X| < 2^229. The
// functions use only compiler builtins, so the same text also compiles for
// the host, where a test checks them against exact integers.
#pragma once

#include <stdint.h>

#ifndef OZFP4_HD
#define OZFP4_HD __device__ __forceinline__
#endif

namespace ozfp4 {

// acc += (-1)^neg (m 2^sh) modulo 2^256, m = m0 + m1 2^64 + m2 2^128,
// 0 <= sh < 128
OZFP4_HD void add_shifted256(uint64_t (&acc)[4], uint64_t m0, uint64_t m1, uint64_t m2, bool neg,
                             int sh) {
  const int ws = sh >> 6, bs = sh & 63;
  const uint64_t in[4] = {m0, m1, m2, 0};
  uint64_t t[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = i - ws;                    // source word
    const uint64_t lo = (j >= 0 && j < 4) ? in[j] : 0;
    const uint64_t below = (j - 1 >= 0 && j - 1 < 4) ? in[j - 1] : 0;
    t[i] = bs ? ((lo << bs) | (below >> (64 - bs))) : lo;
  }
  if (neg) {   // two's complement: invert and add one
    uint64_t c = 1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint64_t v = ~t[i] + c;
      c = (c && v == 0) ? 1 : 0;
      t[i] = v;
    }
  }
  uint64_t carry = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint64_t s = acc[i] + t[i];
    const uint64_t c1 = s < acc[i] ? 1 : 0;
    const uint64_t s2 = s + carry;
    const uint64_t c2 = s2 < s ? 1 : 0;
    acc[i] = s2;
    carry = c1 | c2;
  }
}

// RN_even(x 2^e2) for the 256-bit two's-complement x, including subnormal
// results and overflow to infinity; 0 gives +0.0
OZFP4_HD double round_scaled256(const uint64_t (&x)[4], int e2) {
  uint64_t w[4] = {x[0], x[1], x[2], x[3]};
  const bool neg = (int64_t)w[3] < 0;
  if (neg) {
    uint64_t c = 1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint64_t v = ~w[i] + c;
      c = (c && v == 0) ? 1 : 0;
      w[i] = v;
    }
  }
  int n = 0;   // bit length of |x|
#pragma unroll
  for (int i = 3; i >= 0; --i)
    if (n == 0 && w[i]) n = 64 * i + 64 - __builtin_clzll((unsigned long long)w[i]);
  if (n == 0) return 0.0;
  const int E = n - 1 + e2;
  double r;
  if (E > 1023) {
    r = __builtin_huge_val();
  } else {
    const int qe = (E - 52 > -1074 ? E - 52 : -1074);
    const int sh = qe - e2;   // bits of |x| below the result's quantum
    if (sh <= 0) {
      r = __builtin_ldexp((double)w[0], e2);   // |x| < 2^53: exact
    } else {
      // the 64 bits of |x| from bit sh up, the bit below them, and whether
      // any lower bit is set
      auto word = [&](int i) { return (i >= 0 && i < 4) ? w[i] : 0ull; };
      const int ws = sh >> 6, bs = sh & 63;
      uint64_t Rm = bs ? ((word(ws) >> bs) | (word(ws + 1) << (64 - bs))) : word(ws);
      const int b = sh - 1;
      const int rb = (int)((word(b >> 6) >> (b & 63)) & 1ull);
      bool sticky = false;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int lo = 64 * i;
        if (lo + 64 <= b) sticky |= w[i] != 0;
        else if (lo < b) sticky |= (w[i] & ((1ull << (b - lo)) - 1)) != 0;
      }
      if (rb && (sticky || (Rm & 1ull))) ++Rm;
      r = __builtin_ldexp((double)Rm, qe);   // Rm <= 2^53: exact, or +inf
    }
  }
  return neg ? -r : r;
}

}  // namespace ozfp4
