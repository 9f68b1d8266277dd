// Final reduction of Ozaki scheme I (Sec. IV): the exact integer product
// x = sum_h 2197^h H_h from the partial sums of the block anti-diagonals
// (2197 = 13^3: one block pairs three limbs of A with three limbs of B), and
// its single rounding RN(x 2^e2). Compiler builtins and 64-bit integer
// arithmetic only, so the same text also compiles for the host, where a test
// checks it against exact integer arithmetic.
#pragma once

#include <stdint.h>

#include "crt_round.hpp"

namespace ozfp4 {

constexpr int kOziMaxGroups = 9;   // anti-diagonals of 5 x 5 blocks (15 limbs)

OZFP4_HD uint64_t mulhi_u64(uint64_t a, uint64_t b) {
  return (uint64_t)(((unsigned __int128)a * b) >> 64);
}

// x = sum_{h < nh} 2197^h H[h] by Horner's rule from the top group, in
// 192-bit two's complement (the value stays below 2^131 in magnitude for
// k <= 2^17, so no step wraps), then RN(x 2^e2) with sign.
OZFP4_HD double ozi_compose_round(const int64_t (&H)[kOziMaxGroups], int nh, int e2) {
  uint64_t w0 = (uint64_t)H[nh - 1];
  uint64_t w1 = (uint64_t)(H[nh - 1] >> 63);
  uint64_t w2 = w1;
#pragma unroll
  for (int h = kOziMaxGroups - 2; h >= 0; --h) {
    if (h > nh - 2) continue;
    // (w2 w1 w0) *= 2197, modulo 2^192
    const uint64_t h0 = mulhi_u64(w0, 2197u), h1 = mulhi_u64(w1, 2197u);
    w0 *= 2197u;
    const uint64_t t1 = w1 * 2197u;
    w1 = t1 + h0;
    w2 = w2 * 2197u + h1 + (w1 < h0 ? 1u : 0u);
    // += H[h], sign-extended to 192 bits
    const uint64_t a0 = (uint64_t)H[h], ext = (uint64_t)(H[h] >> 63);
    const unsigned __int128 s0 = (unsigned __int128)w0 + a0;
    const unsigned __int128 s1 = (unsigned __int128)w1 + ext + (uint64_t)(s0 >> 64);
    w0 = (uint64_t)s0;
    w1 = (uint64_t)s1;
    w2 = w2 + ext + (uint64_t)(s1 >> 64);
  }
  const bool neg = (int64_t)w2 < 0;
  if (neg) {   // two's-complement negation
    w0 = ~w0 + 1;
    const uint64_t c0 = (w0 == 0) ? 1 : 0;
    w1 = ~w1 + c0;
    const uint64_t c1 = (c0 && w1 == 0) ? 1 : 0;
    w2 = ~w2 + c1;
  }
  return round_scaled(w0, w1, w2, e2, neg);
}

}  // namespace ozfp4
