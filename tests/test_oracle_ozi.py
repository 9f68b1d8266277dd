"""Pins of the Ozaki-scheme-I oracle (oracle/ozaki1_fp4.py, Sec. IV) against
what the paper and the mathematics fix: the printed limb counts and bounds,
the lemma's gap-free boundary, brute-force limb and group sums, the limb
expansion identity, correctly rounded results on exactly convertible inputs,
and the paper's statement that schemes I and II give bitwise the same C on
the same converted inputs (Sec. VII-A)."""

from fractions import Fraction

import numpy as np
import pytest

import oracle as o
from paper_2608_06812_amd.workloads import dgemm_inputs, paper_law_inputs


def test_capacity_matches_printed_limb_counts(paper):
    lc = paper["limb_counts"]
    # FP64 significand (53 bits) fits in 15 limbs, FP32 (24) in 7, INT8 in 3
    assert o.ozi_capacity(lc["fp64"]) == 53
    assert o.ozi_capacity(lc["fp64"] - 1) < 53
    assert o.ozi_capacity(lc["fp32"]) >= 24
    assert o.ozi_capacity(lc["fp32"] - 1) < 24
    assert o.ozi_capacity(lc["int8"]) >= 8
    assert o.ozi_capacity(lc["int8"] - 1) < 8
    # Lemma 1: X_1 = 4, X_2 = 56, X_3 = 732 -> 2, 5, 9 bits
    assert [o.ozi_capacity(p) for p in (1, 2, 3)] == [
        x.bit_length() - 1 for x in paper["gap_free_ranges"]]
    with pytest.raises(ValueError):
        o.ozi_capacity(16)


def test_limbs_equal_scalar_greedy_and_reconstruct(paper):
    rng = np.random.default_rng(7)
    S = set(paper["doubled_set"])
    for p in (1, 3, 7, 15):
        X = o.gap_free_range(p)
        lim = min(X, 1 << 53)
        vals = list(rng.integers(-lim, lim + 1, size=300)) + [0, 1, -1, lim, -lim, X if X < 2**62 else 0]
        Xi = np.array(vals, dtype=np.int64)
        a = o.ozi_limbs(Xi, p)
        for idx, v in enumerate(vals):
            want = o.limb_decompose(int(v), p)
            got = [int(a[i][idx]) for i in range(p)]
            assert got == want
            assert sum(c * 13 ** i for i, c in enumerate(got)) == int(v)
            assert all(c in S and abs(c) <= paper["greedy_max_limb"] for c in got)


@pytest.mark.parametrize("p", [1, 2, 3, 7, 14])
def test_limbs_gap_free_boundary(p):
    """Lemma 1: every |N| <= X_p has p greedy limbs; X_p + 1 does not."""
    X = o.gap_free_range(p)
    o.ozi_limbs(np.array([X, -X]), p)
    with pytest.raises(ValueError):
        o.ozi_limbs(np.array([X + 1]), p)
    with pytest.raises(ValueError):
        o.ozi_limbs(np.array([-X - 1]), p)


def test_group_products_brute_force(paper):
    rng = np.random.default_rng(8)
    p = 4
    a = [rng.choice(paper["doubled_set"], size=(3, 5)).astype(np.int64) for _ in range(p)]
    b = [rng.choice(paper["doubled_set"], size=(5, 2)).astype(np.int64) for _ in range(p)]
    G = o.ozi_group_products(a, b)
    assert len(G) == 2 * p - 1
    for g in range(2 * p - 1):
        for i in range(3):
            for j in range(2):
                want = 0
                for u in range(p):
                    for v in range(p):
                        if u + v == g:
                            want += sum(int(a[u][i, q]) * int(b[v][q, j]) for q in range(5))
                assert int(G[g][i, j]) == want


def test_fp64_configuration_counts(paper):
    """15 x 15 limbs: 225 products in 29 anti-diagonal groups, the deepest
    with 15 pairs, whose FP32 accumulation is exact up to K = 17,476."""
    p = paper["limb_counts"]["fp64"]
    sizes = [sum(1 for i in range(p) if 0 <= g - i < p) for g in range(2 * p - 1)]
    assert sum(sizes) == paper["ozi_fp64_gemms"] and len(sizes) == 29 and max(sizes) == 15
    K = paper["lemma2_greedy_group_bound"]
    assert o.fp32_exact_bound(K, 8, max(sizes)) and not o.fp32_exact_bound(K + 1, 8, max(sizes))


@pytest.mark.parametrize("p", [15, 9, 7])
def test_expansion_equals_integer_product(p):
    """Eq. (expand): sum_g 13^g G_g is the exact product of the converted
    operands (Python-int matmul), including entries at the capacity."""
    A, B = dgemm_inputs(9, 7, 33, 2.0, 11 + p)
    A[0, 3] = -A[0, :].max() * 1.75
    res = o.dgemm_ozi(A, B, p)
    assert np.all(res["x"] == o.exact_int_matmul(res["Ai"], res["Bi"]))
    assert np.abs(res["Ai"]).max() <= 2 ** res["c"]


def test_definition_brute_force():
    """C_ij = RN(sum_q A~_iq B~_qj 2^-(s_i + t_j)) with the conversion done
    in exact rationals and Python-int sums (tiny, wide exponent range)."""
    rng = np.random.default_rng(12)
    for trial in range(4):
        m, n, k = 3, 4, 6
        A = (rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-40, 40, size=(m, k)))
        B = (rng.random((k, n)) - 0.5) * np.exp2(rng.integers(-40, 40, size=(k, n)))
        if trial == 3:
            A[1, :] = 0.0
            B[:, 2] *= 1e-300
        res = o.dgemm_ozi(A, B, 15)
        c = 53
        s = o.shift_exponents(A, axis=1, c=c)
        t = o.shift_exponents(B, axis=0, c=c)
        Ai = o.to_integers_fraction(A, s, axis=1)
        Bi = o.to_integers_fraction(B, t, axis=0)
        for i in range(m):
            for j in range(n):
                acc = sum(int(Ai[i, q]) * int(Bi[q, j]) for q in range(k))
                want = float(Fraction(acc) / Fraction(2) ** (int(s[i]) + int(t[j])))
                assert res["C"][i, j] == want


def test_exactly_convertible_inputs_are_rounded_once():
    """When every entry of a row of A (column of B) is an integer multiple of
    the line's lowest unit, the conversion is exact and C is the correctly
    rounded exact product (phi = 0 in the paper's law is such a case)."""
    A, B = paper_law_inputs(6, 5, 40, 0, 3)
    # (1 + u) 2^0 with 52-bit u: representable exactly with c = 53
    res = o.dgemm_ozi(A, B, 15)
    for i in range(6):
        for j in range(5):
            assert res["C"][i, j] == float(o.exact_product_entry(A, B, i, j))


@pytest.mark.parametrize("shape,phi,seed", [((17, 13, 50), 0.5, 1), ((8, 9, 300), 4.0, 2),
                                            ((5, 6, 7), 16.0, 3)])
def test_schemes_agree_bitwise(shape, phi, seed):
    """Sec. VII-A: with the same converted inputs (c = 53 for both operands)
    schemes I and II compute the same exact integer product and round it
    once, so C agrees bit for bit."""
    m, n, k = shape
    A, B = dgemm_inputs(m, n, k, phi, seed)
    assert o.capacity_bits(k, o.select_moduli(18)) == (53, 53)
    c2 = o.dgemm(A, B, 18)
    c1 = o.dgemm_ozi(A, B, 15)
    assert np.array_equal(c1["Ai"], c2["Ai"]) and np.array_equal(c1["Bi"], c2["Bi"])
    assert np.all(c1["x"] == c2["x"])
    assert np.array_equal(c1["C"].view(np.uint64), c2["C"].view(np.uint64))


def test_sub_block_selection():
    A, B = dgemm_inputs(20, 11, 30, 1.0, 5)
    full = o.dgemm_ozi(A, B, 15)
    rows, cols = np.array([0, 7, 19]), np.array([10, 2])
    part = o.dgemm_ozi(A, B, 15, rows=rows, cols=cols)
    assert np.array_equal(part["C"], full["C"][np.ix_(rows, cols)])
