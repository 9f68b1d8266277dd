// Host-side constants of the method, derived at library initialisation from
// the definitions in the paper (nothing is typed in):
//   * the two-limb moduli and their greedy pairwise-coprime order (Sec. V-A);
//   * P, the CRT weights w_l = M_l (M_l^{-1} mod m_l) and their 42-bit
//     chunks (Sec. V-B);
//   * the capacity split (c_A, c_B) for an inner dimension k (Sec. IV-B with
//     Eq. (crt));
//   * the canonical two-limb split of every residue and its E2M1 codes
//     (Sec. III, Sec. V-A), and for the Karatsuba moduli the split whose
//     limb sum is representable too, as lookup tables for the encoder;
//   * the three greedy limbs of every int8 (Sec. III).
#pragma once

#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <vector>

namespace ozfp4 {

constexpr int kMaxModuli = 27;   // the greedy list: the printed 19, then 47, 43, 41, 31, 29, 19, 17, 11

// ---- minimal unsigned multiword integer (little-endian 32-bit words) ----
struct Big {
  static constexpr int W = 8;  // 256 bits: P < 2^129 for 20 moduli
  uint32_t w[W];
  Big() { std::memset(w, 0, sizeof(w)); }
  explicit Big(uint64_t v) {
    std::memset(w, 0, sizeof(w));
    w[0] = (uint32_t)v;
    w[1] = (uint32_t)(v >> 32);
  }
  void mul_small(uint32_t f) {
    uint64_t carry = 0;
    for (int i = 0; i < W; ++i) {
      uint64_t t = (uint64_t)w[i] * f + carry;
      w[i] = (uint32_t)t;
      carry = t >> 32;
    }
  }
  // divides in place, returns the remainder
  uint32_t div_small(uint32_t d) {
    uint64_t rem = 0;
    for (int i = W - 1; i >= 0; --i) {
      uint64_t cur = (rem << 32) | w[i];
      w[i] = (uint32_t)(cur / d);
      rem = cur % d;
    }
    return (uint32_t)rem;
  }
  void sub_one() {
    for (int i = 0; i < W; ++i) {
      if (w[i]-- != 0) break;
    }
  }
  int bitlen() const {
    for (int i = W - 1; i >= 0; --i)
      if (w[i]) return 32 * i + 32 - __builtin_clz(w[i]);
    return 0;
  }
  // bits [lo, lo + n) as an integer, n <= 52
  uint64_t bits(int lo, int n) const {
    uint64_t out = 0;
    for (int b = 0; b < n; ++b) {
      int pos = lo + b;
      if (pos >= 32 * W) break;
      out |= (uint64_t)((w[pos >> 5] >> (pos & 31)) & 1u) << b;
    }
    return out;
  }
};

// ---- Sec. III: E2M1 codes of doubled values, greedy digits ----
inline int e2m1_code_of_limb(int c) {
  // stored value c/2; magnitudes 0, .5, 1, 1.5, 2, 3, 4, 6 -> codes 0..7
  int a = c < 0 ? -c : c;
  int code;
  switch (a) {
    case 0: code = 0; break;
    case 1: code = 1; break;
    case 2: code = 2; break;
    case 3: code = 3; break;
    case 4: code = 4; break;
    case 6: code = 5; break;
    case 8: code = 6; break;
    case 12: code = 7; break;
    default: return -1;
  }
  return (c < 0) ? (code | 8) : code;
}

// greedy digit: smallest-magnitude representative mod 13, +-5 -> -+8 (Lemma 2)
inline int greedy13(int x) {
  int s = ((x + 6) % 13 + 13) % 13 - 6;
  if (s == 5) return -8;
  if (s == -5) return 8;
  return s;
}

inline bool limb_in_S(int c) { return e2m1_code_of_limb(c) >= 0; }

// ---- Sec. V-A: two-limb moduli and the greedy list ----
// every two-limb modulus up to 400, descending
inline std::vector<int> two_limb_moduli_desc() {
  static const int S[] = {-12, -8, -6, -4, -3, -2, -1, 0, 1, 2, 3, 4, 6, 8, 12};
  std::vector<int> two_limb;
  for (int m = 400; m >= 2; --m) {
    std::vector<char> seen(m, 0);
    int count = 0;
    for (int a : S)
      for (int b : S) {
        int r = ((a + 13 * b) % m + m) % m;
        if (!seen[r]) { seen[r] = 1; ++count; }
      }
    if (count == m) two_limb.push_back(m);
  }
  return two_limb;
}

// the greedy choice of Sec. V-A seeded with `seed`: descending over the
// two-limb moduli, each pick coprime to every modulus chosen so far, until
// kMaxModuli moduli (the seed first)
inline std::vector<int> greedy_seeded(const std::vector<int>& seed) {
  std::vector<int> chosen = seed;
  for (int m : two_limb_moduli_desc()) {
    if ((int)chosen.size() >= kMaxModuli) break;
    bool ok = true;
    for (int q : chosen) {
      int a = m, b = q;
      while (b) { int t = a % b; a = b; b = t; }
      if (a != 1) { ok = false; break; }
    }
    if (ok) chosen.push_back(m);
  }
  return chosen;
}

inline std::vector<int> greedy_moduli() { return greedy_seeded({}); }

// canonical two-limb split of residue r in [0, m): returns false if none
inline bool two_limb_split(int r, int m, int* c0, int* c1) {
  int rp = r;
  if (2 * rp > m) rp -= m;
  int cands[2] = {rp, rp > 0 ? rp - m : rp + m};
  for (int cand : cands) {
    int a = greedy13(cand);
    int q = (cand - a) / 13;  // exact
    int b = greedy13(q);
    if ((((a + 13 * b - r) % m) + m) % m == 0) {
      *c0 = a;
      *c1 = b;
      return true;
    }
  }
  return false;
}

// Sec. V-A, Karatsuba: every class of m has limbs c0, c1 in S whose sum
// c0 + c1 is in S as well
inline bool is_karatsuba(int m) {
  static const int S[] = {-12, -8, -6, -4, -3, -2, -1, 0, 1, 2, 3, 4, 6, 8, 12};
  std::vector<char> seen(m, 0);
  int count = 0;
  for (int a : S)
    for (int b : S) {
      if (!limb_in_S(a + b)) continue;
      int r = ((a + 13 * b) % m + m) % m;
      if (!seen[r]) { seen[r] = 1; ++count; }
    }
  return count == m;
}

// limbs of residue r for a Karatsuba modulus: c0, c1, c0 + c1 in S, all
// within +-8; the canonical split when it qualifies, else the qualifying
// split with the smallest |c1|, then the smallest |c0|
inline bool sum_limb_split(int r, int m, int* c0, int* c1) {
  auto ok = [](int c) { return limb_in_S(c) && c >= -8 && c <= 8; };
  int a, b;
  if (two_limb_split(r, m, &a, &b) && ok(a + b)) {
    *c0 = a;
    *c1 = b;
    return true;
  }
  bool found = false;
  int best1 = 0, best0 = 0;
  for (int y = -8; y <= 8; ++y) {
    if (!ok(y)) continue;
    for (int x = -8; x <= 8; ++x) {
      if (!ok(x) || !ok(x + y) || (((x + 13 * y - r) % m) + m) % m != 0) continue;
      const bool better = !found || std::abs(y) < std::abs(best1) ||
                          (std::abs(y) == std::abs(best1) && std::abs(x) < std::abs(best0));
      if (better) { found = true; best1 = y; best0 = x; }
    }
  }
  *c0 = best0;
  *c1 = best1;
  return found;
}

// One-limb moduli (an extension of Sec. V-A): every class of m holds an
// element of S, so one limb represents each residue (c1 = 0) and the
// residue product is one limb product. A list with h one-limb heads starts
// with the first h of 11, 9, 8, 7, 5 (pairwise coprime) and continues by the
// greedy rule seeded with them; h = 1 is 11 followed by the greedy list
// (11 is coprime to its first 26 moduli).
constexpr int kMaxHeads = 5;
constexpr int kOneLimbHeads[kMaxHeads] = {11, 9, 8, 7, 5};

// the element of S congruent to r mod m of smallest magnitude, the positive
// one on a tie; false if there is none
inline bool one_limb_split(int r, int m, int* c) {
  static const int S[] = {0, 1, -1, 2, -2, 3, -3, 4, -4, 6, -6, 8, -8, 12, -12};
  for (int v : S)   // ascending magnitude, positive first
    if ((((v - r) % m) + m) % m == 0) {
      *c = v;
      return true;
    }
  return false;
}

// ---- device-side constant blocks (plain data, copied once per device) ----
struct ModConst {
  int m[kMaxModuli];
  int ksum[kMaxModuli];      // index among the Karatsuba moduli of the list, or -1
  int lut_off[kMaxModuli];   // start of modulus l in the encoder LUT (entries)
  double inv[kMaxModuli];    // fl(1 / m)
  double md[kMaxModuli];     // m as double
};

// Chunk width of the exact FP64 CRT sums. With R = sum (m_l - 1) <= 1983
// for up to 27 moduli, R (2^42 - 1) < 2^53, so every chunk sum
// sum r_l w_l,c, every q P_c with q <= R, and every carry-normalised chunk
// is an integer below 2^53 and exact in FP64. Three chunks (126 bits) cover
// P for up to 19 moduli (P < 2^124), four (168 bits) up to 27 (P < 2^162).
constexpr int kCrtChunkBits = 42;

struct CrtConst {
  int L;
  int nc;                    // chunks in use: 3 while P < 2^126, else 4
  double W[kMaxModuli][4];   // 42-bit chunks of w_l
  double Pc[4];              // 42-bit chunks of P
  double Qc[4];              // ~ 2^(42 c) / P, weights of the quotient estimate
  double sym_limit;          // ~ (P / 2)(1 - 2^-30): a rounded |x| below it is inside (-P/2, P/2]
  uint64_t P[3];             // P as a 192-bit integer
};

struct HostTables {
  std::vector<int> moduli;                 // 20, greedy order
  ModConst mod;
  CrtConst crt[kMaxModuli + 1];            // index L (2..27)
  std::vector<uint16_t> lut;               // encoder LUT, all 20 moduli
  std::vector<uint32_t> lut_k;             // encoder LUT of the Karatsuba mode
  int nk[kMaxModuli + 1];                  // Karatsuba moduli among the first L
  uint16_t lut8[256];                      // int8 -> three limb codes
  Big P[kMaxModuli + 1];                   // product of the first L moduli
  // the lists with h = 1..kMaxHeads one-limb heads (index h; 0 unused)
  struct List {
    std::vector<int> moduli;               // kMaxModuli, heads first
    ModConst mod;                          // the whole list (encoder)
    ModConst tail;                         // the two-limb moduli after the heads (residue GEMM)
    ModConst head;                         // the heads (single-product GEMM)
    std::vector<uint16_t> lut;             // encoder LUT of the whole list
    CrtConst crt[kMaxModuli + 1];
    Big P[kMaxModuli + 1];
  } lists[kMaxHeads + 1];
  bool ok = false;
};

// P and the CRT constants of every prefix of a moduli list (Sec. V-B)
inline bool build_crt(const std::vector<int>& moduli, CrtConst* crt, Big* P) {
  for (int L = 0; L <= kMaxModuli; ++L) {
    std::memset(&crt[L], 0, sizeof(CrtConst));
    P[L] = Big(1);
    if (L < 1) continue;
    for (int l = 0; l < L; ++l) P[L].mul_small((uint32_t)moduli[l]);
    CrtConst& c = crt[L];
    c.L = L;
    const int B = kCrtChunkBits;
    c.nc = P[L].bitlen() <= 3 * B ? 3 : 4;
    if (P[L].bitlen() > c.nc * B) return false;
    double Pd = 0.0;
    for (int q = 0; q < 4; ++q) {
      c.Pc[q] = (double)P[L].bits(B * q, B);
      Pd += std::ldexp(c.Pc[q], B * q);
    }
    for (int q = 0; q < 4; ++q) c.Qc[q] = std::ldexp(1.0 / Pd, B * q);
    c.sym_limit = 0.5 * Pd * (1.0 - std::ldexp(1.0, -30));
    for (int q = 0; q < 3; ++q) c.P[q] = P[L].bits(64 * q, 32) | (P[L].bits(64 * q + 32, 32) << 32);
    for (int l = 0; l < L; ++l) {
      int m = moduli[l];
      Big Mi = P[L];
      Mi.div_small((uint32_t)m);          // exact: M_l = P / m_l
      Big tmp = Mi;
      uint32_t Mmod = tmp.div_small((uint32_t)m);
      int u = -1;
      for (int x = 1; x < m; ++x)
        if ((uint64_t)Mmod * x % m == 1) { u = x; break; }
      if (u < 0) return false;
      Big w = Mi;
      w.mul_small((uint32_t)u);           // w_l = M_l u_l < P
      for (int q = 0; q < 4; ++q) c.W[l][q] = (double)w.bits(B * q, B);
    }
  }
  return true;
}

// Encoder LUT of modulus m: 3m entries, index r + m for a remainder
// estimate r in [-m, 2m) of a signed integer x; entry = code(c0) |
// code(c1) << 8 for the canonical split of the class of x mod m. The LUT of
// the Karatsuba mode has the same indexing and 32-bit entries code(c0) |
// code(c1) << 8 | code(c0 + c1) << 16 from the sum-limb split of a Karatsuba
// modulus (the canonical split and a zero sum code for the others).
inline bool build_tables(HostTables& T) {
  T.moduli = greedy_moduli();
  if ((int)T.moduli.size() != kMaxModuli) return false;
  std::memset(&T.mod, 0, sizeof(T.mod));
  int off = 0, nk = 0;
  T.lut.clear();
  T.lut_k.clear();
  T.nk[0] = 0;
  for (int l = 0; l < kMaxModuli; ++l) {
    int m = T.moduli[l];
    const bool kar = is_karatsuba(m);
    T.mod.m[l] = m;
    T.mod.ksum[l] = kar ? nk++ : -1;
    T.nk[l + 1] = nk;
    T.mod.lut_off[l] = off;
    T.mod.inv[l] = 1.0 / (double)m;
    T.mod.md[l] = (double)m;
    for (int ri = -m; ri < 2 * m; ++ri) {
      int cls = ((ri % m) + m) % m;
      int c0, c1;
      if (!two_limb_split(cls, m, &c0, &c1)) return false;
      int k0 = e2m1_code_of_limb(c0), k1 = e2m1_code_of_limb(c1);
      if (k0 < 0 || k1 < 0) return false;
      T.lut.push_back((uint16_t)(k0 | (k1 << 8)));
      if (kar) {
        if (!sum_limb_split(cls, m, &c0, &c1)) return false;
        k0 = e2m1_code_of_limb(c0);
        k1 = e2m1_code_of_limb(c1);
      }
      const int ks = kar ? e2m1_code_of_limb(c0 + c1) : 0;
      if (k0 < 0 || k1 < 0 || ks < 0) return false;
      T.lut_k.push_back((uint32_t)k0 | ((uint32_t)k1 << 8) | ((uint32_t)ks << 16));
    }
    off += 3 * m;
  }
  // int8: three greedy limbs (X_3 = 732 >= 128)
  for (int v = -128; v < 128; ++v) {
    int rest = v, codes = 0;
    for (int i = 0; i < 3; ++i) {
      int c = greedy13(rest);
      int code = e2m1_code_of_limb(c);
      if (code < 0) return false;
      codes |= code << (4 * i);
      rest = (rest - c) / 13;
    }
    if (rest != 0) return false;
    T.lut8[v + 128] = (uint16_t)codes;
  }
  if (!build_crt(T.moduli, T.crt, T.P)) return false;

  // the lists with one-limb heads: the heads' one-limb codes (second limb
  // 0), the two-limb moduli's canonical splits
  for (int h = 1; h <= kMaxHeads; ++h) {
    HostTables::List& Ls = T.lists[h];
    Ls.moduli = greedy_seeded(std::vector<int>(kOneLimbHeads, kOneLimbHeads + h));
    if ((int)Ls.moduli.size() != kMaxModuli) return false;
    std::memset(&Ls.mod, 0, sizeof(ModConst));
    std::memset(&Ls.tail, 0, sizeof(ModConst));
    std::memset(&Ls.head, 0, sizeof(ModConst));
    Ls.lut.clear();
    int off1 = 0;
    for (int l = 0; l < kMaxModuli; ++l) {
      const int m = Ls.moduli[l];
      ModConst& part = l < h ? Ls.head : Ls.tail;
      const int pl = l < h ? l : l - h;
      for (ModConst* mc : {&Ls.mod, &part}) {
        const int i = mc == &Ls.mod ? l : pl;
        mc->m[i] = m;
        mc->ksum[i] = -1;
        mc->lut_off[i] = off1;
        mc->inv[i] = 1.0 / (double)m;
        mc->md[i] = (double)m;
      }
      for (int ri = -m; ri < 2 * m; ++ri) {
        const int cls = ((ri % m) + m) % m;
        int c0, c1 = 0;
        if (l < h) {
          if (!one_limb_split(cls, m, &c0)) return false;
        } else if (!two_limb_split(cls, m, &c0, &c1)) {
          return false;
        }
        const int k0 = e2m1_code_of_limb(c0), k1 = e2m1_code_of_limb(c1);
        if (k0 < 0 || k1 < 0) return false;
        Ls.lut.push_back((uint16_t)(k0 | (k1 << 8)));
      }
      off1 += 3 * m;
    }
    if (!build_crt(Ls.moduli, Ls.crt, Ls.P)) return false;
  }
  T.ok = true;
  return true;
}

// Largest b with 2 k 2^b < P (Eq. (crt)) and the split c_A = min(cmax,
// ceil(b/2)), c_B = min(cmax, b - c_A) (Sec. IV-B); cmax = 53 is the
// paper's rule, up to 63 the wide-range extension. Returns false if b < 2.
inline bool capacity_split(const Big& P, int64_t k, int cmax, int* cA, int* cB) {
  if (k < 1) return false;
  // 2 k 2^b < P  <=>  2^(b+1) <= floor((P - 1) / k)
  Big q = P;
  q.sub_one();
  q.div_small((uint32_t)k);
  int b = q.bitlen() - 2;
  if (b < 2) return false;
  int a = std::min(cmax, (b + 1) / 2);
  *cA = a;
  *cB = std::min(cmax, b - a);
  return true;
}

}  // namespace ozfp4
