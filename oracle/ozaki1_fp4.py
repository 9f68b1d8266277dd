"""Plain, slow, exact CPU oracle for Ozaki scheme I on FP4 (E2M1) limbs.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the CPU
baseline of the benchmark, never by the product path.

Follows Sec. IV of the paper (the FP4 adaptation of Ozaki scheme I): each
converted operand is written positionally in base 13 with greedy limbs in S
(Lemma 1), the product expands into p q limb products <a_i, b_j> weighted by
13^(i+j) (Eq. (expand)), products with the same i + j are summed into one
group, and the groups are combined by one weighted sum; the result is rounded
once after the inverse scaling (Sec. IV-B).

Readings (the GPU library documents the same ones):
  * capacity c = floor(log2 min(X_p, 2^53)) bits for both operands
    (Sec. IV-B), so p = 15 gives c = 53, the capacity Ozaki scheme II uses
    whenever its c_A = c_B = 53;
  * integer conversion and final rounding as in scheme II (round half to
    even; one round-to-nearest-even of x 2^-(s_i + t_j), subnormals and
    overflow included).
"""

from __future__ import annotations

import numpy as np

from .ozaki2_fp4 import (_limb_matmul, gap_free_range, round_scaled, shift_exponents,
                         to_integers)

__all__ = ["ozi_capacity", "ozi_limbs", "ozi_group_products", "ozi_compose", "dgemm_ozi",
           "OZI_MAX_LIMBS"]

#: The FP64 configuration of the paper: p = q = 15 limbs, 225 limb products.
OZI_MAX_LIMBS = 15


def ozi_capacity(p: int) -> int:
    """c = floor(log2 min(X_p, 2^53)) (Sec. IV-B)."""
    if not 1 <= p <= OZI_MAX_LIMBS:
        raise ValueError("p must be in [1, 15]")
    return min(gap_free_range(p), 1 << 53).bit_length() - 1


def ozi_limbs(Xi: np.ndarray, p: int) -> list[np.ndarray]:
    """Greedy base-13 limbs a_0..a_{p-1} of every entry of the integer array
    Xi, with Xi = sum_i 13^i a_i (Lemma 1). Each step takes the class
    representative of smallest magnitude, with the +-5 classes taking -+8
    (Lemma 2), and divides the exact remainder by 13."""
    rest = np.asarray(Xi, dtype=np.int64).copy()
    out = []
    for _ in range(p):
        s = np.mod(rest + 6, 13) - 6               # smallest representative, in [-6, 6]
        c = np.where(s == 5, -8, np.where(s == -5, 8, s))
        out.append(c.astype(np.int64))
        rest = (rest - c) // 13                    # exact: rest - c is a multiple of 13
    if np.any(rest != 0):
        raise ValueError(f"entries need more than {p} greedy limbs")
    return out


def ozi_group_products(a: list[np.ndarray], b: list[np.ndarray]) -> list[np.ndarray]:
    """G_g = sum_{i + j = g} <a_i, b_j> for g = 0 .. p + q - 2 (Eq. (expand)
    grouped along anti-diagonals), each an exact int64 matrix."""
    p, q = len(a), len(b)
    G = []
    for g in range(p + q - 1):
        acc = None
        for i in range(p):
            j = g - i
            if 0 <= j < q:
                t = _limb_matmul(a[i], b[j])
                acc = t if acc is None else acc + t
        G.append(acc)
    return G


def ozi_compose(G: list[np.ndarray]) -> np.ndarray:
    """x = sum_g 13^g G_g in Python ints (object array): the exact integer
    product of the converted operands."""
    x = np.zeros(G[0].shape, dtype=object)
    for g, Gg in enumerate(G):
        x = x + Gg.astype(object) * (13 ** g)
    return x


def dgemm_ozi(A: np.ndarray, B: np.ndarray, p: int = OZI_MAX_LIMBS, rows=None,
              cols=None) -> dict:
    """C = A B by Ozaki scheme I on base-13 E2M1 limbs with p = q limbs
    (Sec. IV). `rows` / `cols` restrict the output to a sub-block (the
    scaling still reads whole rows of A and whole columns of B). Returns the
    capacity c, shifts s and t, converted integers, limbs, group sums G, the
    exact integer product x and C (FP64)."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    m, k = A.shape
    k2, n = B.shape
    assert k == k2
    rows = np.arange(m) if rows is None else np.asarray(rows)
    cols = np.arange(n) if cols is None else np.asarray(cols)
    c = ozi_capacity(p)
    As, Bs = A[rows, :], B[:, cols]
    s = shift_exponents(As, axis=1, c=c)
    t = shift_exponents(Bs, axis=0, c=c)
    Ai = to_integers(As, s, axis=1)
    Bi = to_integers(Bs, t, axis=0)
    a = ozi_limbs(Ai, p)
    b = ozi_limbs(Bi, p)
    G = ozi_group_products(a, b)
    x = ozi_compose(G)
    C = np.empty((len(rows), len(cols)), dtype=np.float64)
    for i in range(len(rows)):
        for j in range(len(cols)):
            C[i, j] = round_scaled(x[i, j], int(s[i]) + int(t[j]))
    return {"c": c, "s": s, "t": t, "Ai": Ai, "Bi": Bi, "a": a, "b": b, "G": G, "x": x, "C": C}
