"""Plain, slow, exact CPU oracle for FP64 matrix multiplication by Ozaki
scheme II on FP4 (E2M1) limbs with a two-term split of the converted
operands: the second route of the wide-range extension.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the CPU
baseline of the benchmark, never by the product path.

The conversion of Sec. IV-B shares one exponent per row of A (column of B):
A~ = round(A 2^s) keeps c bits measured from the line's largest element, so
an element many binades below it loses its low bits. This is the
quantization error the paper names for wide exponent ranges. The two-term
split keeps what the first conversion rounds away as a second integer:

    A 2^s = A1 + 2^-d A2 + e,   A1 = RNE(A 2^s),
    A2 = RNE((A 2^s - A1) 2^d),  |e| <= 2^(-d-1),

and the same for B with its column shifts t. With d = min(c_A, c_B),

    (A1 + 2^-d A2)(B1 + 2^-d B2) = 2^-2d (2^2d X11 + 2^d X12 + X22),
    X11 = A1 B1,  X12 = A1 B2 + A2 B1,  X22 = A2 B2.

Each X is an exact integer matrix product that scheme II computes through
its residue route with the same L moduli, X12 as one product over the
concatenated k ([A1 | A2] times [B2 ; B1]). All three lie inside the
symmetric CRT range: |A1| <= 2^c_A, |A2| <= 2^(d-1), so
|X12| <= k 2^(d-1) (2^c_A + 2^c_B) <= k 2^(c_A + c_B), which the capacity
rule (2 k 2^(c_A + c_B) < P) keeps below P / 2, like |X11| and |X22|. Then

    C = RN((2^2d X11 + 2^d X12 + X22) 2^-(s + t + 2d)),

one rounding of the exact product of the split operands. An element whose
significand lies within c_A + d bits of its line's largest element is held
exactly, so inputs whose lines span fewer than about c_A + d - 53 binades
give the correctly rounded product fl(AB).

Readings (the paper describes only the one-term conversion): d =
min(c_A, c_B), so both cross terms share one scale and one residue product;
the three products use the same moduli and capacities as the one-term
method; the conversion of each term rounds half to even. With one-limb
heads (``heads`` > 0, see one_limb_fp4) the moduli are that list's and the
heads take the single limb product.
"""

from __future__ import annotations

from fractions import Fraction

import numpy as np

from .one_limb_fp4 import residue_products_one_limb, select_moduli_one_limb
from .ozaki2_fp4 import (capacity_bits, crt_reconstruct, residue_products, round_scaled,
                         select_moduli, shift_exponents)

__all__ = ["split_terms", "split_terms_fraction", "split_scale", "dgemm_split2",
           "dgemm_split2_definition"]


def split_scale(cA: int, cB: int) -> int:
    """d, the binary scale of the second terms: min(c_A, c_B)."""
    return min(cA, cB)


def split_terms_fraction(X: np.ndarray, shifts: np.ndarray, axis: int, d: int):
    """(X1, X2) by exact rational arithmetic: X1 = RNE(X 2^s),
    X2 = RNE((X 2^s - X1) 2^d), one shift per row (axis=1) or per column
    (axis=0). Returns two object arrays of Python ints."""
    X = np.asarray(X, dtype=np.float64)
    X1 = np.empty(X.shape, dtype=object)
    X2 = np.empty(X.shape, dtype=object)
    for idx in np.ndindex(X.shape):
        s = int(shifts[idx[0]] if axis == 1 else shifts[idx[1]])
        v = Fraction(float(X[idx])) * Fraction(2) ** s
        a1 = round(v)                               # half to even
        X1[idx] = a1
        X2[idx] = round((v - a1) * Fraction(2) ** d)
    return X1, X2


def split_terms(X: np.ndarray, shifts: np.ndarray, axis: int, d: int):
    """Same result as ``split_terms_fraction``, vectorised in FP64, as int64.

    T = X 2^s is exact unless it falls below 2^-1022, where both terms are 0
    either way (|T 2^d| < 2^-959 < 1/2). X1 = rint(T) rounds half to even;
    T - X1 is exact (the fraction of T, or 0 once |T| >= 2^52), and so is
    its product by 2^d (at most 2^(d-1) in magnitude); rint rounds it."""
    X = np.asarray(X, dtype=np.float64)
    sh = (shifts[:, None] if axis == 1 else shifts[None, :]).astype(np.int64)
    T = np.ldexp(X, sh)
    X1 = np.rint(T)
    X2 = np.rint(np.ldexp(T - X1, d))
    return X1.astype(np.int64), X2.astype(np.int64)


def _moduli(n_moduli: int, heads: int) -> list[int]:
    return select_moduli_one_limb(n_moduli, heads) if heads else select_moduli(n_moduli)


def _residue_route(Xi: np.ndarray, Yi: np.ndarray, moduli, heads: int = 0) -> tuple[list, np.ndarray]:
    """Residues of Xi Yi for every modulus (the scheme-II residue products of
    Sec. V-A; the single limb product for one-limb heads) and the symmetric
    CRT reconstruction (Sec. V-B)."""
    one = set(moduli[:min(heads, len(moduli))])
    res = [(residue_products_one_limb if m in one else residue_products)(Xi, Yi, m)["r"]
           for m in moduli]
    return res, crt_reconstruct(res, moduli)


def dgemm_split2(A: np.ndarray, B: np.ndarray, n_moduli: int, rows=None, cols=None,
                 cmax: int = 53, heads: int = 0) -> dict:
    """C = A B by scheme II with the two-term split (see the module text).

    Optional `rows` / `cols` restrict the output to a block (shifts still
    come from whole rows of A and columns of B). Returns the moduli,
    capacities, d, shifts, the four term matrices, the residues and exact
    integers of the three products, the combined integer X and C."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    m, k = A.shape
    assert B.shape[0] == k
    rows = np.arange(m) if rows is None else np.asarray(rows)
    cols = np.arange(B.shape[1]) if cols is None else np.asarray(cols)
    moduli = _moduli(n_moduli, heads)
    cA, cB = capacity_bits(k, moduli, cmax)
    d = split_scale(cA, cB)
    As, Bs = A[rows, :], B[:, cols]
    s = shift_exponents(As, axis=1, c=cA)
    t = shift_exponents(Bs, axis=0, c=cB)
    A1, A2 = split_terms(As, s, axis=1, d=d)
    B1, B2 = split_terms(Bs, t, axis=0, d=d)
    r11, X11 = _residue_route(A1, B1, moduli, heads)
    r12, X12 = _residue_route(np.hstack([A1, A2]), np.vstack([B2, B1]), moduli, heads)
    r22, X22 = _residue_route(A2, B2, moduli, heads)
    X = np.empty(X11.shape, dtype=object)
    C = np.empty(X11.shape, dtype=np.float64)
    for i in range(X.shape[0]):
        for j in range(X.shape[1]):
            X[i, j] = (int(X11[i, j]) << (2 * d)) + (int(X12[i, j]) << d) + int(X22[i, j])
            C[i, j] = round_scaled(X[i, j], int(s[i]) + int(t[j]) + 2 * d)
    return {"moduli": moduli, "cA": cA, "cB": cB, "d": d, "s": s, "t": t,
            "A1": A1, "A2": A2, "B1": B1, "B2": B2,
            "r11": r11, "r12": r12, "r22": r22, "X11": X11, "X12": X12, "X22": X22,
            "X": X, "C": C}


def dgemm_split2_definition(A: np.ndarray, B: np.ndarray, n_moduli: int,
                            cmax: int = 53, heads: int = 0) -> np.ndarray:
    """The defined result without residues: C_ij = RN(sum_k (A1 + 2^-d A2)_ik
    (B1 + 2^-d B2)_kj 2^-(s_i + t_j)), terms from exact rationals, sums of
    Python ints (tiny inputs)."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    m, k = A.shape
    n = B.shape[1]
    moduli = _moduli(n_moduli, heads)
    cA, cB = capacity_bits(k, moduli, cmax)
    d = split_scale(cA, cB)
    s = shift_exponents(A, axis=1, c=cA)
    t = shift_exponents(B, axis=0, c=cB)
    A1, A2 = split_terms_fraction(A, s, axis=1, d=d)
    B1, B2 = split_terms_fraction(B, t, axis=0, d=d)
    C = np.empty((m, n), dtype=np.float64)
    for i in range(m):
        for j in range(n):
            acc = 0   # in units of 2^-2d
            for q in range(k):
                a = (int(A1[i, q]) << d) + int(A2[i, q])
                b = (int(B1[q, j]) << d) + int(B2[q, j])
                acc += a * b
            C[i, j] = round_scaled(acc, int(s[i]) + int(t[j]) + 2 * d)
    return C
