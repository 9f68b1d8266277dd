"""Ozaki scheme II with a one-limb modulus: an extension of the moduli choice
of Sec. V-A, for the CPU oracle.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the CPU
baseline of the benchmark, never by the product path.

Sec. V-A admits a modulus when every residue class has a two-limb
representative c0 + 13 c1 with c0, c1 in S, and picks them greedily,
largest first, pairwise coprime. A modulus whose every class already holds
an element of S needs only c1 = 0: one limb per operand, so its residue
product is the single limb product a0 b0 instead of four. Such one-limb
moduli are small (2..9, 11, 13); 11 is the only one coprime to the greedy
list's first 26 moduli (it is the greedy rule's own 27th pick).

Reading of this extension (the paper does not use it; the GPU library
documents the same one):
  * with h one-limb heads (0 <= h <= 5), the list of n moduli starts with
    the first min(h, n) of 11, 9, 8, 7, 5 (pairwise coprime one-limb
    moduli, each taking one product) and continues by the greedy rule of
    Sec. V-A over the two-limb moduli, seeded with those heads: descending,
    each pick coprime to every modulus chosen so far; h = 0 is the greedy
    list, h = 1 is 11 followed by the first n - 1 greedy moduli;
    2 <= n <= 27;
  * the one-limb representative of a residue r mod m is the element of S
    congruent to r of smallest magnitude, the positive one on a tie;
  * everything else is scheme II unchanged: capacities from P by the same
    rule (here P = 11 P_{n-1}), the same shifts, integer conversion, CRT and
    one rounding; for FP32 inputs the FP32 emulation's capacities and its
    one rounding to binary32.
"""

from __future__ import annotations

import math

import numpy as np

from .ozaki2_fp4 import (capacity_bits, crt_reconstruct, doubled_set, exact_int_matmul,
                         residue_products, residues, round_scaled, shift_exponents,
                         to_integers, to_integers_fraction, two_limb_moduli)
from .sgemm_fp4 import capacity_bits_fp32, round_scaled_f32

__all__ = [
    "is_one_limb_modulus", "one_limb_moduli", "ONE_LIMB_MODULUS", "ONE_LIMB_HEADS",
    "select_moduli_one_limb",
    "one_limb_split", "one_limb_table", "one_limb_plane", "residue_products_one_limb",
    "dgemm_one_limb", "dgemm_one_limb_definition", "sgemm_one_limb",
]

#: The one-limb modulus of the extension.
ONE_LIMB_MODULUS = 11

#: The one-limb heads, in the order a list takes them.
ONE_LIMB_HEADS = (11, 9, 8, 7, 5)


def is_one_limb_modulus(m: int) -> bool:
    """Every residue class mod m holds an element of S (one limb, c1 = 0)."""
    return m >= 2 and len({c % m for c in doubled_set()}) == m


def one_limb_moduli(limit: int = 64) -> list[int]:
    """All one-limb moduli 2 <= m <= limit, found exhaustively."""
    return [m for m in range(2, limit + 1) if is_one_limb_modulus(m)]


def select_moduli_one_limb(L: int, heads: int = 1) -> list[int]:
    """The first min(heads, L) of 11, 9, 8, 7, 5, then the greedy rule of
    Sec. V-A over the two-limb moduli seeded with them, L moduli in all."""
    if not 2 <= L <= 27:
        raise ValueError("the one-limb list has 2..27 moduli")
    if not 0 <= heads <= len(ONE_LIMB_HEADS):
        raise ValueError("0..5 one-limb heads")
    chosen = list(ONE_LIMB_HEADS[:min(heads, L)])
    for m in sorted(two_limb_moduli(), reverse=True):
        if len(chosen) == L:
            break
        if all(math.gcd(m, q) == 1 for q in chosen):
            chosen.append(m)
    if len(chosen) != L:
        raise ValueError(f"only {len(chosen)} coprime moduli exist")
    return chosen


def _heads_of(moduli, heads: int) -> set:
    return set(moduli[:min(heads, len(moduli))])


def one_limb_split(r: int, m: int) -> int:
    """The element of S congruent to r mod m of smallest magnitude (the
    positive one on a tie)."""
    cands = [c for c in doubled_set() if (c - r) % m == 0]
    if not cands:
        raise ValueError(f"residue {r} has no one-limb representative mod {m}")
    return min(cands, key=lambda c: (abs(c), -c))


def one_limb_table(m: int) -> list[int]:
    """The one-limb representative of every residue r in [0, m)."""
    return [one_limb_split(r, m) for r in range(m)]


def one_limb_plane(Xi: np.ndarray, m: int) -> np.ndarray:
    """The limb plane c0 of X~ mod m, elementwise."""
    tab = np.array(one_limb_table(m), dtype=np.int64)
    return tab[residues(Xi, m)]


def residue_products_one_limb(Ai: np.ndarray, Bi: np.ndarray, m: int) -> dict:
    """The residue product of a one-limb modulus: a = a0 and b = b0 (mod m),
    so the product is the single limb product G0 = a0 b0, r = G0 mod m."""
    a0 = one_limb_plane(Ai, m)
    b0 = one_limb_plane(Bi, m)
    k = a0.shape[1]
    assert 36 * k < (1 << 53)
    G0 = np.rint(a0.astype(np.float64) @ b0.astype(np.float64)).astype(np.int64)
    return {"G0": G0, "r": np.mod(G0, m)}


def dgemm_one_limb(A: np.ndarray, B: np.ndarray, n_moduli: int, rows=None, cols=None,
                   check_definition: bool = False, cmax: int = 53, heads: int = 1) -> dict:
    """C = A B by scheme II over the list of select_moduli_one_limb: the
    one-limb product for the heads, the four-product two-limb route for the
    others (Sec. V-A, Sec. VI-D), the CRT and one rounding (Sec. V-B).

    rows / cols restrict the output to a block (the shifts still come from
    whole lines). With check_definition=True the reconstructed integers are
    compared with the exact product of the converted operands."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    m, k = A.shape
    assert B.shape[0] == k
    n = B.shape[1]
    rows = np.arange(m) if rows is None else np.asarray(rows)
    cols = np.arange(n) if cols is None else np.asarray(cols)
    moduli = select_moduli_one_limb(n_moduli, heads)
    one = _heads_of(moduli, heads)
    cA, cB = capacity_bits(k, moduli, cmax)
    As, Bs = A[rows, :], B[:, cols]
    s = shift_exponents(As, axis=1, c=cA)
    t = shift_exponents(Bs, axis=0, c=cB)
    Ai = to_integers(As, s, axis=1)
    Bi = to_integers(Bs, t, axis=0)
    assert np.all(np.abs(Ai) <= (1 << cA)) and np.all(np.abs(Bi) <= (1 << cB))
    res = [(residue_products_one_limb if q in one else residue_products)(Ai, Bi, q)["r"]
           for q in moduli]
    x = crt_reconstruct(res, moduli)
    if check_definition:
        assert np.all(exact_int_matmul(Ai, Bi) == x), "CRT reconstruction differs from the exact product"
    C = np.empty((len(rows), len(cols)), dtype=np.float64)
    for i in range(len(rows)):
        for j in range(len(cols)):
            C[i, j] = round_scaled(x[i, j], int(s[i]) + int(t[j]))
    return {"moduli": moduli, "cA": cA, "cB": cB, "s": s, "t": t, "Ai": Ai, "Bi": Bi,
            "r": res, "x": x, "C": C}


def dgemm_one_limb_definition(A: np.ndarray, B: np.ndarray, n_moduli: int,
                              cmax: int = 53, heads: int = 1) -> np.ndarray:
    """The defined result without the residue route, capacities from the
    one-limb list's P: C_ij = RN(sum_k A~_ik B~_kj 2^-(s_i+t_j)) by
    Python-int sums (tiny inputs)."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    m, k = A.shape
    n = B.shape[1]
    cA, cB = capacity_bits(k, select_moduli_one_limb(n_moduli, heads), cmax)
    s = shift_exponents(A, axis=1, c=cA)
    t = shift_exponents(B, axis=0, c=cB)
    Ai = to_integers_fraction(A, s, axis=1)
    Bi = to_integers_fraction(B, t, axis=0)
    C = np.empty((m, n), dtype=np.float64)
    for i in range(m):
        for j in range(n):
            acc = sum(int(Ai[i, q]) * int(Bi[q, j]) for q in range(k))
            C[i, j] = round_scaled(acc, int(s[i]) + int(t[j]))
    return C


def sgemm_one_limb(A: np.ndarray, B: np.ndarray, n_moduli: int, rows=None, cols=None,
                   heads: int = 1) -> dict:
    """C = A B for FP32 A, B by the FP32 emulation over the one-limb list:
    the FP32 capacities c_A = min(24, ceil(b/2)), c_B = min(24, b - c_A)
    from the list's P, the one-limb product for 11, and one rounding of the
    exact product to binary32."""
    A = np.asarray(A, dtype=np.float32).astype(np.float64)
    B = np.asarray(B, dtype=np.float32).astype(np.float64)
    m, k = A.shape
    assert B.shape[0] == k
    n = B.shape[1]
    rows = np.arange(m) if rows is None else np.asarray(rows)
    cols = np.arange(n) if cols is None else np.asarray(cols)
    moduli = select_moduli_one_limb(n_moduli, heads)
    one = _heads_of(moduli, heads)
    cA, cB = capacity_bits_fp32(k, moduli)
    As, Bs = A[rows, :], B[:, cols]
    s = shift_exponents(As, axis=1, c=cA)
    t = shift_exponents(Bs, axis=0, c=cB)
    Ai = to_integers(As, s, axis=1)
    Bi = to_integers(Bs, t, axis=0)
    res = [(residue_products_one_limb if q in one else residue_products)(Ai, Bi, q)["r"]
           for q in moduli]
    x = crt_reconstruct(res, moduli)
    C = np.empty((len(rows), len(cols)), dtype=np.float32)
    for i in range(len(rows)):
        for j in range(len(cols)):
            C[i, j] = round_scaled_f32(x[i, j], int(s[i]) + int(t[j]))
    return {"moduli": moduli, "cA": cA, "cB": cB, "s": s, "t": t, "Ai": Ai, "Bi": Bi,
            "r": res, "x": x, "C": C}
