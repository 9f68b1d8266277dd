// Exact direct CRT reconstruction of one element and its single final
// rounding (Sec. V-B), shared by the CRT kernel. The functions use only
// compiler builtins, so the same text also compiles for the host, where a
// test checks them against exact rational arithmetic.
#pragma once

#include <stdint.h>

#include "tables.hpp"

#ifndef OZFP4_HD
#define OZFP4_HD __device__ __forceinline__
#endif

namespace ozfp4 {

OZFP4_HD uint64_t bits_of(double x) { return __builtin_bit_cast(uint64_t, x); }
OZFP4_HD double double_of(uint64_t b) { return __builtin_bit_cast(double, b); }

OZFP4_HD uint64_t word3(uint64_t w0, uint64_t w1, uint64_t w2, int i) {
  return i == 0 ? w0 : (i == 1 ? w1 : (i == 2 ? w2 : 0ull));
}

// low 64 bits of (w >> sh), sh >= 1
OZFP4_HD uint64_t shr3(uint64_t w0, uint64_t w1, uint64_t w2, int sh) {
  if (sh >= 192) return 0;
  const int ws = sh >> 6, bs = sh & 63;
  const uint64_t lo = word3(w0, w1, w2, ws), hi = word3(w0, w1, w2, ws + 1);
  return bs ? ((lo >> bs) | (hi << (64 - bs))) : lo;
}

OZFP4_HD int bit3(uint64_t w0, uint64_t w1, uint64_t w2, int b) {
  if (b >= 192) return 0;
  return (int)((word3(w0, w1, w2, b >> 6) >> (b & 63)) & 1ull);
}

// any of bits [0, b) set
OZFP4_HD bool below3(uint64_t w0, uint64_t w1, uint64_t w2, int b) {
  if (b <= 0) return false;
  if (b >= 192) return (w0 | w1 | w2) != 0;
  const int ws = b >> 6, bs = b & 63;
  uint64_t acc = 0;
  if (ws > 0) acc |= w0;
  if (ws > 1) acc |= w1;
  const uint64_t part = word3(w0, w1, w2, ws);
  if (bs) acc |= part & ((1ull << bs) - 1);
  return acc != 0;
}

// RN_even(M * 2^e2) for the 192-bit magnitude M, with sign
OZFP4_HD double round_scaled(uint64_t w0, uint64_t w1, uint64_t w2, int e2,
                                               bool neg) {
  if ((w0 | w1 | w2) == 0) return 0.0;
  const int n = w2 ? 192 - __builtin_clzll((unsigned long long)w2)
                   : (w1 ? 128 - __builtin_clzll((unsigned long long)w1) : 64 - __builtin_clzll((unsigned long long)w0));
  const int E = n - 1 + e2;
  double r;
  if (E > 1023) {
    r = __builtin_huge_val();
  } else {
    const int qe = (E - 52 > -1074 ? E - 52 : -1074);
    const int sh = qe - e2;
    if (sh <= 0) {
      r = __builtin_ldexp((double)w0, e2);  // M < 2^53: exact
    } else {
      uint64_t Rm = shr3(w0, w1, w2, sh);
      const int rb = bit3(w0, w1, w2, sh - 1);
      const bool st = below3(w0, w1, w2, sh - 1);
      if (rb && (st || (Rm & 1ull))) ++Rm;
      r = __builtin_ldexp((double)Rm, qe);  // Rm <= 2^53: exact or +inf
    }
  }
  return neg ? -r : r;
}

// Exact path. x' = S - q P is assembled from the 42-bit chunk differences
// v_c = sig_c - q P_c (exact integers below 2^53 in magnitude) as a 192-bit
// two's-complement integer and mapped into the symmetric range (-P/2, P/2];
// crt_symmetric returns |x| in (w0, w1, w2) and whether x < 0. s3 = 0 when
// three chunks are in use (then P_3 = 0).
OZFP4_HD bool crt_symmetric(double s0, double s1, double s2, double s3, double q,
                            const CrtConst* __restrict__ cc, uint64_t* o0, uint64_t* o1,
                            uint64_t* o2) {
  const int64_t v0 = (int64_t)__builtin_fma(-q, cc->Pc[0], s0);
  const int64_t v1 = (int64_t)__builtin_fma(-q, cc->Pc[1], s1);
  const int64_t v2 = (int64_t)__builtin_fma(-q, cc->Pc[2], s2);
  const int64_t v3 = (int64_t)__builtin_fma(-q, cc->Pc[3], s3);
  constexpr int64_t MASK = (1ll << kCrtChunkBits) - 1;
  const int64_t d0 = v0 & MASK;
  int64_t t = v1 + (v0 >> 42);
  const int64_t d1 = t & MASK;
  t = v2 + (t >> 42);
  const int64_t d2 = t & MASK;
  const int64_t t3 = v3 + (t >> 42);
  // x' = d0 + d1 2^42 + d2 2^84 + t3 2^126
  uint64_t w0 = (uint64_t)d0 | ((uint64_t)d1 << 42);
  uint64_t w1 = ((uint64_t)d1 >> 22) | ((uint64_t)d2 << 20) | ((uint64_t)t3 << 62);
  uint64_t w2 = (uint64_t)(t3 >> 2);
  bool neg = (int64_t)w2 < 0;
  if (neg) {  // two's-complement negation of the 192-bit value
    w0 = ~w0 + 1;
    const uint64_t c0 = (w0 == 0) ? 1 : 0;
    w1 = ~w1 + c0;
    const uint64_t c1 = (c0 && w1 == 0) ? 1 : 0;
    w2 = ~w2 + c1;
  }
  // symmetric range: x -> x -+ P when 2|x| > P (or 2|x| == P and x < 0)
  const uint64_t x0 = w0 << 1, x1 = (w1 << 1) | (w0 >> 63), x2 = (w2 << 1) | (w1 >> 63);
  int cmp = (x2 != cc->P[2]) ? (x2 > cc->P[2] ? 1 : -1)
          : (x1 != cc->P[1]) ? (x1 > cc->P[1] ? 1 : -1)
          : (x0 != cc->P[0]) ? (x0 > cc->P[0] ? 1 : -1) : 0;
  if (cmp > 0 || (cmp == 0 && neg)) {
    const uint64_t n0 = cc->P[0] - w0;
    const uint64_t b0 = cc->P[0] < w0 ? 1 : 0;
    const uint64_t n1 = cc->P[1] - w1 - b0;
    const uint64_t b1 = (cc->P[1] < w1 || (cc->P[1] == w1 && b0)) ? 1 : 0;
    const uint64_t n2 = cc->P[2] - w2 - b1;
    w0 = n0; w1 = n1; w2 = n2;
    neg = !neg;
  }
  *o0 = w0;
  *o1 = w1;
  *o2 = w2;
  return neg;
}

// RN(x 2^e2) of the exact symmetric x, including subnormal results and
// overflow to infinity.
OZFP4_HD double crt_exact(double s0, double s1, double s2, double s3, double q,
                          const CrtConst* __restrict__ cc, int e2) {
  uint64_t w0, w1, w2;
  const bool neg = crt_symmetric(s0, s1, s2, s3, q, cc, &w0, &w1, &w2);
  return round_scaled(w0, w1, w2, e2, neg);
}

// Fast path for three chunks, in FP64 only. Carry normalisation gives
// x' = t 2^84 + d1 2^42 + d0 with 0 <= d0, d1 < 2^42, every step exact.
//   |t| <= 2: (t 2^42 + d1) is exact, so one FMA rounds x' once.
//   |t| >= 3: |x'| >= 2^85. y = d1 2^42 + d0 is rounded to odd at 53 bits
//     (Fast2Sum gives the sign of the error), a grid of at most 2^31 that is
//     at least 4 times finer than the grid of x' (>= 2^33); adding t 2^84
//     and rounding to nearest then equals RN(x') (rounding to odd with two
//     extra bits, Boldo and Melquiond).
// RN(x' 2^e2) = RN(x') 2^e2 whenever the result is normal. The path gives up
// (returns false) when |x'| may lie outside (-P/2, P/2], which the quotient
// estimate leaves only when S / P is within about 2^-30 of a half-integer,
// or when the result may be subnormal; crt_exact then decides.
OZFP4_HD bool crt_fast3(double s0, double s1, double s2, double q,
                                          const CrtConst* __restrict__ cc, int e2, double* out) {
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
  const double r_small = __builtin_fma(__builtin_fma(t, kC, d1), kC, d0);
  const double D1 = d1 * kC;
  const double sy = D1 + d0;
  const double ey = d0 - (sy - D1);
  uint64_t bits = (uint64_t)bits_of(sy);
  bits = ey > 0.0 ? (bits | 1ull) : ((ey < 0.0 && !(bits & 1ull)) ? bits - 1ull : bits);
  const double r_large = __builtin_fma(t, 0x1p84, double_of(bits));
  const double r = __builtin_fabs(t) <= 2.0 ? r_small : r_large;
  if (!(__builtin_fabs(r) < cc->sym_limit)) return false;
  if (r != 0.0) {
    int fe;
    (void)__builtin_frexp(r, &fe);
    if (fe + e2 <= -1020) return false;
  }
  *out = __builtin_ldexp(r, e2);
  return true;
}

}  // namespace ozfp4
