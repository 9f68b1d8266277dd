"""Pins of the two-term split oracle (oracle/split2_fp4.py), the second
wide-range route: each check ties it to something other than itself.

* The split against its definition by exact rational arithmetic, its error
  bound |A 2^s - A1 - 2^-d A2| <= 2^(-d-1), the term bounds that keep all
  three products inside the CRT range, and exact representation of every
  element within c + d bits of its line's largest one.
* The residue route (three scheme-II products, X12 over the concatenated k,
  combined in integers and rounded once) against the direct expansion of
  the split operands' product in Python integers, on tiny matrices with
  very wide exponent spreads and few moduli (so that the second terms carry
  many bits), and the three exact integers against Python-int products.
* Inputs whose lines span fewer than c + d - 53 binades are held exactly,
  so C must equal fl(AB), the exact product rounded once: the paper's input
  law at phi = 32 (Sec. VII-A) and the wide-range law of the phi = 4
  workload restricted to such a span.
* On the phi = 4 law itself the normalized error falls from the one-term
  method's 2^-31..2^-36 to within the final rounding (<= 2^-52).
* Planted mistakes (a cross term at the wrong scale, the concatenation in
  the wrong order, the second term at the wrong scale, X22 dropped) are each
  caught by the residue-route pin.
* With one-limb heads: the same route against its definition over the
  list, and at k = 32768 the four-head 21-moduli list's C equal bit for bit
  to the 19 greedy moduli's."""

import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as o
import oracle.split2_fp4 as s2
from paper_2608_06812_amd.workloads import dgemm_inputs, paper_law_inputs


def _wide(m, k, spread, seed):
    rng = np.random.default_rng(seed)
    X = (rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-spread, spread + 1, (m, k)))
    X[rng.random((m, k)) < 0.1] = 0.0
    return X


@pytest.mark.parametrize("d", [8, 26, 53, 63])
def test_split_terms_match_the_rational_definition_and_bound(d):
    A = _wide(7, 40, 300, 1)
    A[2, :] = 0.0                               # a zero row
    A[3, 5] = 5e-324                            # the smallest subnormal
    A[4, :] = np.ldexp(A[4, :], -1000)          # a row of tiny values
    s = o.shift_exponents(A, axis=1, c=min(d, 53))
    X1, X2 = o.split_terms(A, s, axis=1, d=d)
    F1, F2 = o.split_terms_fraction(A, s, axis=1, d=d)
    assert np.array_equal(X1.astype(object), F1) and np.array_equal(X2.astype(object), F2)
    for i, q in np.ndindex(A.shape):
        v = Fraction(float(A[i, q])) * Fraction(2) ** int(s[i])
        err = v - int(X1[i, q]) - Fraction(int(X2[i, q]), 2 ** d)
        assert abs(err) <= Fraction(1, 2 ** (d + 1))
        assert abs(int(X1[i, q])) <= 2 ** min(d, 53) and abs(int(X2[i, q])) <= 2 ** (d - 1)


def test_elements_within_c_plus_d_bits_are_held_exactly():
    """A row whose elements all lie within c + d - 53 binades of its
    largest one: A 2^s = A1 + 2^-d A2 exactly, for every element."""
    c, d = 53, 53
    rng = np.random.default_rng(3)
    A = (1 + rng.random((6, 50))) * np.exp2(-rng.integers(0, c + d - 53, (6, 50)))
    A[:, 0] = 1.0                               # the row maximum sits at 2^0
    s = o.shift_exponents(A, axis=1, c=c)
    X1, X2 = o.split_terms(A, s, axis=1, d=d)
    for i, q in np.ndindex(A.shape):
        v = Fraction(float(A[i, q])) * Fraction(2) ** int(s[i])
        assert v == int(X1[i, q]) + Fraction(int(X2[i, q]), 2 ** d)


@pytest.mark.parametrize("L,cmax,spread,seed", [
    (2, 53, 40, 1), (3, 53, 60, 2), (4, 53, 300, 3), (6, 53, 20, 4),
    (10, 53, 100, 5), (19, 53, 200, 6), (23, 63, 200, 7), (27, 63, 600, 8)])
def test_residue_route_equals_the_expanded_definition(L, cmax, spread, seed):
    rng = np.random.default_rng(seed)
    for _ in range(6):
        m, n, k = (int(x) for x in rng.integers(1, 6, 3))
        A, B = _wide(m, k, spread, rng.integers(1 << 30)), _wide(k, n, spread, rng.integers(1 << 30))
        try:
            res = o.dgemm_split2(A, B, L, cmax=cmax)
        except ValueError:          # too few moduli for this k
            continue
        want = o.dgemm_split2_definition(A, B, L, cmax=cmax)
        assert np.array_equal(res["C"].view(np.int64), want.view(np.int64))
        # the three reconstructions are the exact integer products
        A1 = res["A1"].astype(object)
        A2 = res["A2"].astype(object)
        B1 = res["B1"].astype(object)
        B2 = res["B2"].astype(object)
        assert np.array_equal(res["X11"], A1.dot(B1))
        assert np.array_equal(res["X12"], A1.dot(B2) + A2.dot(B1))
        assert np.array_equal(res["X22"], A2.dot(B2))


@pytest.mark.parametrize("h,L,spread,seed", [(1, 12, 60, 11), (5, 21, 200, 12), (4, 21, 40, 13),
                                          (3, 8, 100, 14)])
def test_residue_route_with_one_limb_heads(h, L, spread, seed):
    """With one-limb heads (11, 9, 8, 7, 5 first) the split route equals its
    expanded definition over that list, and the three reconstructions are
    the exact integer products."""
    rng = np.random.default_rng(seed)
    for _ in range(4):
        m, n, k = (int(x) for x in rng.integers(1, 6, 3))
        A, B = _wide(m, k, spread, rng.integers(1 << 30)), _wide(k, n, spread, rng.integers(1 << 30))
        res = o.dgemm_split2(A, B, L, heads=h)
        assert res["moduli"] == o.select_moduli_one_limb(L, heads=h)
        want = o.dgemm_split2_definition(A, B, L, heads=h)
        assert np.array_equal(res["C"].view(np.int64), want.view(np.int64))
        A1, A2 = res["A1"].astype(object), res["A2"].astype(object)
        B1, B2 = res["B1"].astype(object), res["B2"].astype(object)
        assert np.array_equal(res["X11"], A1.dot(B1))
        assert np.array_equal(res["X12"], A1.dot(B2) + A2.dot(B1))
        assert np.array_equal(res["X22"], A2.dot(B2))


def test_four_heads_give_the_greedy_19_result_at_k_32768():
    """At k = 32768 the 21-moduli list with four heads has the capacities of
    the 19 greedy moduli (53 / 53), so the split route's C is the same bit
    for bit."""
    rng = np.random.default_rng(15)
    k = 32768
    A = (rng.random((3, k)) - 0.5) * np.exp(4.0 * rng.standard_normal((3, k)))
    B = (rng.random((k, 2)) - 0.5) * np.exp(4.0 * rng.standard_normal((k, 2)))
    g = o.dgemm_split2(A, B, 19)
    h = o.dgemm_split2(A, B, 21, heads=4)
    assert (g["cA"], g["cB"]) == (h["cA"], h["cB"]) == (53, 53)
    assert np.array_equal(g["C"].view(np.int64), h["C"].view(np.int64))


def test_products_stay_inside_the_crt_range_at_the_capacity_bound():
    """Largest possible terms at the largest k each moduli count allows:
    k 2^(c_A + c_B) and the cross-term bound stay below P / 2."""
    for L in range(2, 28):
        ms = o.select_moduli(L)
        P = o.moduli_product(ms)
        for cmax in (53, 63):
            for k in (1, 100, 16384, 65536):
                try:
                    cA, cB = o.capacity_bits(k, ms, cmax)
                except ValueError:
                    continue
                d = s2.split_scale(cA, cB)
                assert 2 * k * 2 ** (cA + cB) < P
                assert 2 * k * (2 ** (cA + d - 1) + 2 ** (d - 1 + cB)) < P
                assert 2 * k * 2 ** (2 * d - 2) < P


def _correctly_rounded(A, B):
    ex, _ = o.exact_block(A, B, np.arange(A.shape[0]), np.arange(B.shape[1]))
    return np.array([[float(ex[i, j]) for j in range(ex.shape[1])] for i in range(ex.shape[0])])


def test_paper_law_phi32_is_correctly_rounded():
    """Sec. VII-A's law at phi = 32: every element of a row lies within 33
    binades of the row's largest, so c + d = 106 bits hold it exactly and
    C = fl(AB) bit for bit (the one-term method misses it)."""
    A, B = paper_law_inputs(6, 5, 300, 32, 11)
    C = o.dgemm_split2(A, B, 19)["C"]
    fl = _correctly_rounded(A, B)
    assert np.array_equal(C.view(np.int64), fl.view(np.int64))
    one = o.dgemm(A, B, 19)["C"]
    assert not np.array_equal(one.view(np.int64), fl.view(np.int64))


def test_wide_law_within_the_span_is_correctly_rounded():
    """The phi = 4 law, each line rescaled into a span of 40 binades (far
    above the one-term method's 53 - 1 bits of headroom but inside c + d):
    C = fl(AB)."""
    A, B = dgemm_inputs(5, 6, 400, 4.0, 12)
    for X, axis in ((A, 1), (B, 0)):
        mx = np.max(np.abs(X), axis=axis, keepdims=True)
        np.copyto(X, np.where(np.abs(X) < mx * 2.0 ** -40, np.sign(X) * mx * 2.0 ** -40, X))
    C = o.dgemm_split2(A, B, 19)["C"]
    assert np.array_equal(C.view(np.int64), _correctly_rounded(A, B).view(np.int64))


def test_phi4_accuracy_against_the_one_term_method():
    """The wide-range workload's law (phi = 4) at k = 2048: the normalized
    error (Sec. VII-A metric) of the split is within the final rounding,
    against roughly 2^-31 for the one-term conversion on the same inputs."""
    A, B = dgemm_inputs(6, 6, 2048, 4.0, 13)
    rows = cols = np.arange(6)
    split = o.dgemm_split2(A, B, 19)["C"]
    one = o.dgemm(A, B, 19)["C"]
    e_split = o.normalized_errors_block(split, A, B, rows, cols).max()
    e_one = o.normalized_errors_block(one, A, B, rows, cols).max()
    assert e_split <= 2.0 ** -52
    assert e_one >= 2.0 ** -45 and e_one > 2.0 ** 6 * e_split


# ------------------------------------------------------------- planted mistakes

def _mutant_c(A, B, L, how):
    res = o.dgemm_split2(A, B, L)
    d, s, t = res["d"], res["s"], res["t"]
    X11, X12, X22 = res["X11"], res["X12"], res["X22"]
    A1, A2, B1, B2 = (res[n].astype(object) for n in ("A1", "A2", "B1", "B2"))
    if how == "cross_scale":
        comb = lambda i, j: (int(X11[i, j]) << 2 * d) + (int(X12[i, j]) << (d + 1)) + int(X22[i, j])
    elif how == "concat_order":
        X12w = A1.dot(B1) + A2.dot(B2)
        comb = lambda i, j: (int(X11[i, j]) << 2 * d) + (int(X12w[i, j]) << d) + int(X22[i, j])
    elif how == "no_x22":
        comb = lambda i, j: (int(X11[i, j]) << 2 * d) + (int(X12[i, j]) << d)
    elif how == "second_scale":
        # the second terms taken at scale d + 1 but combined at d
        sA = o.split_terms(A, s, axis=1, d=d + 1)[1].astype(object)
        sB = o.split_terms(B, t, axis=0, d=d + 1)[1].astype(object)
        X12w = A1.dot(sB) + sA.dot(B1)
        X22w = sA.dot(sB)
        comb = lambda i, j: (int(X11[i, j]) << 2 * d) + (int(X12w[i, j]) << d) + int(X22w[i, j])
    C = np.empty(X11.shape)
    for i, j in np.ndindex(C.shape):
        C[i, j] = o.round_scaled(comb(i, j), int(s[i]) + int(t[j]) + 2 * d)
    return C


@pytest.mark.parametrize("how", ["cross_scale", "concat_order", "no_x22", "second_scale"])
def test_planted_mistakes_are_caught(how):
    caught = False
    for seed in range(20):
        rng = np.random.default_rng([77, seed])
        m, n, k = (int(x) for x in rng.integers(2, 6, 3))
        A, B = _wide(m, k, 60, seed), _wide(k, n, 60, seed + 100)
        L = 4
        want = o.dgemm_split2_definition(A, B, L)
        if not np.array_equal(_mutant_c(A, B, L, how).view(np.int64), want.view(np.int64)):
            caught = True
            break
    assert caught, how
