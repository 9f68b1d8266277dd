"""Pins of the one-limb-modulus oracle (oracle/one_limb_fp4.py): each check
ties it to something other than itself.

* Which moduli are one-limb, by brute force over every class; that each is
  also a two-limb modulus (c1 = 0); that 11 is the only one coprime to the
  greedy list's first 26 moduli, and the greedy rule's own 27th pick.
* The one-limb representative of every residue of 11, written out by hand
  from S = {0, +-1, +-2, +-3, +-4, +-6, +-8, +-12}; its E2M1 round trip.
* FP32 exactness of the single limb product at the largest k (bound and an
  adversarial emulated accumulation).
* P and the capacities of the one-limb list against the printed moduli.
* Brute force on tiny matrices: the residue route equals the exact product of
  the converted operands, and C its one rounding; every residue equals the
  exact integer product mod m.
* Integer inputs small enough for every capacity give fl(AB) = the exact
  product, by both lists.
* Lists with h one-limb heads (11, 9, 8, 7, 5): the heads are one-limb and
  pairwise coprime, h = 0 and h = 1 give the greedy list and 11 followed by
  it, the 21-moduli lists with 4 and 5 heads are written out by hand; where
  a list's capacities equal the greedy list's (5 heads and 21 moduli
  against the greedy 18 at k = 16384 and 4096, 4 heads and 21 against the
  greedy 19), C is the same bit for bit; brute force for every h; the
  representatives of 9, 8, 7 and 5 written out by hand; an unseeded tail
  (a two-limb modulus sharing a factor with a head) is caught.
* The FP32 emulation over the list: capacities 24 / 24 at k = 16384 with
  10 moduli, C on tiny matrices against the exact product of the converted
  operands rounded once to binary32 (numpy's single rounding of the exact
  double where that is exact), and small integers giving the exact product.
* Planted mistakes (the two-limb route's c0 used as the one limb, a
  composition weight on the one-limb product, the modulus dropped from the
  list) are each caught."""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle as o
import oracle.one_limb_fp4 as ol

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")


def _printed_moduli():
    with open(GOLDEN) as f:
        return json.load(f)["moduli_L19"]["value"]


def test_one_limb_moduli_by_brute_force():
    S = [0, 1, -1, 2, -2, 3, -3, 4, -4, 6, -6, 8, -8, 12, -12]
    want = [m for m in range(2, 200) if all(any((c - r) % m == 0 for c in S) for r in range(m))]
    assert want == [2, 3, 4, 5, 6, 7, 8, 9, 11, 13]
    assert o.one_limb_moduli(199) == want
    assert all(o.is_two_limb_modulus(m) for m in want)


def test_eleven_is_the_only_coprime_one_limb_modulus():
    greedy26 = o.select_moduli(26)
    assert greedy26[:19] == _printed_moduli()
    free = [m for m in o.one_limb_moduli() if all(math.gcd(m, q) == 1 for q in greedy26)]
    assert free == [11]
    assert o.select_moduli(27)[-1] == 11 and 11 not in greedy26


def test_one_limb_list():
    printed = _printed_moduli()
    assert o.select_moduli_one_limb(18) == [11] + printed[:17]
    assert o.select_moduli_one_limb(2) == [11, 169]
    lst = o.select_moduli_one_limb(27)
    assert len(set(lst)) == 27
    assert all(math.gcd(a, b) == 1 for i, a in enumerate(lst) for b in lst[i + 1:])
    for bad in (1, 28):
        with pytest.raises(ValueError):
            o.select_moduli_one_limb(bad)


def test_one_limb_representatives_of_eleven():
    # 0..4 are in S; 5 = -6 + 11; 6 is in S; 7 = -4 + 11; 8 = -3 + 11 (|-3| < 8);
    # 9 = -2 + 11; 10 = -1 + 11
    assert o.one_limb_table(11) == [0, 1, 2, 3, 4, -6, 6, -4, -3, -2, -1]
    for r, c in enumerate(o.one_limb_table(11)):
        assert (c - r) % 11 == 0
        assert int(2 * o.e2m1_decode(o.e2m1_code(c))) == c
        assert abs(c) <= 6
    for m in o.one_limb_moduli():
        for r in range(m):
            c = o.one_limb_split(r, m)
            assert (c - r) % m == 0 and c in o.doubled_set()


def test_one_limb_product_exact_in_fp32():
    K = o.MAX_K_FP32
    assert o.fp32_exact_bound(K, max_limb=6, terms=1)
    a = np.full(K, 6)
    b = np.full(K, 6)
    assert o.fp32_accumulate_emulated(a, b) == 36 * K
    a[::2] = -6
    assert o.fp32_accumulate_emulated(a, b) == 0
    assert 36 * K < 2 ** 31          # 4 acc converts to int32 exactly


def test_product_and_capacities():
    printed = _printed_moduli()
    P17 = math.prod(printed[:17])
    assert o.moduli_product(o.select_moduli_one_limb(18)) == 11 * P17
    # b is the largest integer with 2 k 2^b < P: log2(11 P17) = 115.07
    assert math.isclose(math.log2(11 * P17), 115.073, abs_tol=1e-3)
    assert o.capacity_bits(16384, o.select_moduli_one_limb(18)) == (50, 50)
    assert o.capacity_bits(4096, o.select_moduli_one_limb(18)) == (51, 51)
    assert o.capacity_bits(16384, o.select_moduli_one_limb(19)) == (53, 52)


def _tiny(seed, m, n, k, spread=30):
    rng = np.random.default_rng(seed)
    A = (rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-spread, spread, (m, k)))
    B = (rng.random((k, n)) - 0.5) * np.exp2(rng.integers(-spread, spread, (k, n)))
    return A, B


@pytest.mark.parametrize("L", [3, 8, 14, 18, 19, 20])
def test_brute_force_tiny(L):
    for seed in range(3):
        A, B = _tiny(100 * L + seed, 3, 4, 6)
        A[1, :] = 0.0
        out = o.dgemm_one_limb(A, B, L, check_definition=True)
        assert out["moduli"][0] == 11
        assert np.array_equal(out["C"], o.dgemm_one_limb_definition(A, B, L))
        exact = o.exact_int_matmul(out["Ai"], out["Bi"])
        for q, r in zip(out["moduli"], out["r"]):
            assert np.array_equal(np.asarray(r, dtype=object), np.mod(exact, q))
        # C is RN of the exact product of the converted operands, scaled
        for i in range(3):
            for j in range(4):
                x = Fraction(int(exact[i, j])) / Fraction(2) ** (int(out["s"][i]) + int(out["t"][j]))
                assert out["C"][i, j] == float(x)


def test_block_restriction_matches_whole():
    A, B = _tiny(7, 9, 8, 40)
    full = o.dgemm_one_limb(A, B, 16)["C"]
    blk = o.dgemm_one_limb(A, B, 16, rows=[1, 4, 8], cols=[0, 7])["C"]
    assert np.array_equal(blk, full[np.ix_([1, 4, 8], [0, 7])])


def test_small_integers_give_the_exact_product_by_both_lists():
    rng = np.random.default_rng(5)
    A = rng.integers(-(1 << 20), 1 << 20, (6, 50)).astype(np.float64)
    B = rng.integers(-(1 << 20), 1 << 20, (50, 5)).astype(np.float64)
    exact = A.astype(object) @ B.astype(object)
    want = np.array([[float(v) for v in row] for row in exact])
    assert np.array_equal(o.dgemm_one_limb(A, B, 18)["C"], want)
    assert np.array_equal(o.dgemm(A, B, 18)["C"], want)


def _mismatch(L=14):
    for seed in range(4):
        A, B = _tiny(900 + seed, 3, 4, 5)
        try:
            got = o.dgemm_one_limb(A, B, L)["C"]
        except (AssertionError, ValueError):
            return True
        if not np.array_equal(got, o.dgemm_one_limb_definition(A, B, L)):
            return True
    return False


def test_unmutated_passes():
    assert not _mismatch()


def test_two_limb_low_limb_as_the_one_limb_is_caught(monkeypatch):
    # the canonical two-limb split of r' = +-5 mod 11 is (-+8, +-1): its low
    # limb alone is not congruent to r
    monkeypatch.setattr(ol, "one_limb_table", lambda m: [o.two_limb_split(r, m)[0] for r in range(m)])
    assert _mismatch()


def test_composition_weight_on_the_one_limb_product_is_caught(monkeypatch):
    orig = ol.residue_products_one_limb

    def bad(Ai, Bi, m):
        out = orig(Ai, Bi, m)
        out["r"] = np.mod(4 * out["G0"], m)
        return out
    monkeypatch.setattr(ol, "residue_products_one_limb", bad)
    assert _mismatch()


def _list_pins_fail():
    lst = ol.select_moduli_one_limb(18)
    return lst != [11] + _printed_moduli()[:17] or o.capacity_bits(16384, lst) != (50, 50)


def test_dropping_the_modulus_is_caught(monkeypatch):
    assert not _list_pins_fail()
    orig = ol.select_moduli_one_limb
    monkeypatch.setattr(ol, "select_moduli_one_limb", lambda L: orig(L)[1:] + [o.select_moduli(L)[-1]])
    assert _list_pins_fail()


def test_sgemm_one_limb_capacities_and_brute_force():
    assert o.capacity_bits_fp32(16384, o.select_moduli_one_limb(10)) == (24, 24)
    assert o.capacity_bits_fp32(16384, o.select_moduli_one_limb(9)) == (22, 21)
    for L in (4, 10, 14):
        for seed in range(3):
            A, B = _tiny(500 + 10 * L + seed, 3, 4, 7, spread=12)
            A, B = A.astype(np.float32), B.astype(np.float32)
            out = o.sgemm_one_limb(A, B, L)
            exact = o.exact_int_matmul(out["Ai"], out["Bi"])
            assert np.all(exact == out["x"])
            for i in range(3):
                for j in range(4):
                    v = Fraction(int(exact[i, j])) / Fraction(2) ** (int(out["s"][i]) + int(out["t"][j]))
                    d = float(v)
                    if Fraction(d) == v:        # exact in FP64: one rounding to binary32
                        assert out["C"][i, j] == np.float32(d)
                    assert out["C"][i, j] == o.round_scaled_f32(int(exact[i, j]),
                                                                int(out["s"][i]) + int(out["t"][j]))


def test_sgemm_one_limb_small_integers_exact():
    rng = np.random.default_rng(8)
    A = rng.integers(-(1 << 10), 1 << 10, (5, 30)).astype(np.float32)
    B = rng.integers(-(1 << 10), 1 << 10, (30, 6)).astype(np.float32)
    exact = A.astype(np.int64) @ B.astype(np.int64)
    assert np.array_equal(o.sgemm_one_limb(A, B, 10)["C"], exact.astype(np.float32))
    assert np.array_equal(o.sgemm(A, B, 10)["C"], exact.astype(np.float32))


def test_heads_are_coprime_one_limb_moduli():
    assert o.ONE_LIMB_HEADS == (11, 9, 8, 7, 5)
    h = o.ONE_LIMB_HEADS
    assert all(o.is_one_limb_modulus(m) for m in h)
    assert all(math.gcd(a, b) == 1 for i, a in enumerate(h) for b in h[i + 1:])
    # 9 * 8 * 7 * 5 = 2520 and 11: no other set of pairwise coprime one-limb
    # moduli (2..9, 11, 13) has a larger product without 13
    assert math.prod(h) == 27720


def test_heads_lists():
    printed = _printed_moduli()
    for L in range(2, 28):
        assert o.select_moduli_one_limb(L, heads=0) == o.select_moduli(L)
        assert o.select_moduli_one_limb(L, heads=1) == [11] + o.select_moduli(L - 1)
    # 5 heads: 115 (5), 112 (7, 2), 111 (3) are skipped by the seeded rule
    assert o.select_moduli_one_limb(21, heads=5) == [
        11, 9, 8, 7, 5, 169, 113, 109, 107, 103, 101, 97, 89, 83, 79, 73, 71, 67, 61, 59, 53]
    assert o.select_moduli_one_limb(21, heads=4) == [
        11, 9, 8, 7, 169, 115, 113, 109, 107, 103, 101, 97, 89, 83, 79, 73, 71, 67, 61, 59, 53]
    assert o.select_moduli_one_limb(3, heads=5) == [11, 9, 8]
    for h in range(6):
        lst = o.select_moduli_one_limb(27, heads=h)
        assert len(set(lst)) == 27
        assert all(math.gcd(a, b) == 1 for i, a in enumerate(lst) for b in lst[i + 1:])
    assert printed[:18] == o.select_moduli(18)
    with pytest.raises(ValueError):
        o.select_moduli_one_limb(18, heads=6)


def test_heads_capacities_match_the_greedy_lists():
    five = o.select_moduli_one_limb(21, heads=5)
    four = o.select_moduli_one_limb(21, heads=4)
    for k in (4096, 16384):
        assert o.capacity_bits(k, five) == o.capacity_bits(k, o.select_moduli(18))
        assert o.capacity_bits(k, four) == o.capacity_bits(k, o.select_moduli(19))
    assert o.capacity_bits(16384, five) == (51, 51)
    assert o.capacity_bits(16384, four) == (53, 53)


def test_representatives_of_the_other_heads():
    assert o.one_limb_table(9) == [0, 1, 2, 3, 4, -4, -3, -2, -1]
    assert o.one_limb_table(8) == [0, 1, 2, 3, 4, -3, -2, -1]
    assert o.one_limb_table(7) == [0, 1, 2, 3, -3, -2, -1]
    assert o.one_limb_table(5) == [0, 1, 2, -2, -1]


@pytest.mark.parametrize("h,L", [(2, 9), (3, 12), (4, 21), (5, 21), (5, 6), (0, 14)])
def test_heads_brute_force_tiny(h, L):
    for seed in range(3):
        A, B = _tiny(700 + 10 * h + seed, 3, 4, 6)
        out = o.dgemm_one_limb(A, B, L, check_definition=True, heads=h)
        assert np.array_equal(out["C"], o.dgemm_one_limb_definition(A, B, L, heads=h))
        exact = o.exact_int_matmul(out["Ai"], out["Bi"])
        for q, r in zip(out["moduli"], out["r"]):
            assert np.array_equal(np.asarray(r, dtype=object), np.mod(exact, q))


def test_same_capacities_give_the_same_c():
    """At k = 16384 the 21-moduli lists with 5 and 4 heads have the
    capacities of the greedy 18 and 19: C is the same bit for bit."""
    rng = np.random.default_rng(12)
    k = 16384
    A = (rng.random((3, k)) - 0.5) * np.exp(0.5 * rng.standard_normal((3, k)))
    B = (rng.random((k, 4)) - 0.5) * np.exp(0.5 * rng.standard_normal((k, 4)))
    g18, g19 = o.dgemm(A, B, 18)["C"], o.dgemm(A, B, 19)["C"]
    assert not np.array_equal(g18, g19)
    assert np.array_equal(o.dgemm_one_limb(A, B, 21, heads=5)["C"].view(np.int64), g18.view(np.int64))
    assert np.array_equal(o.dgemm_one_limb(A, B, 21, heads=4)["C"].view(np.int64), g19.view(np.int64))


def test_unseeded_tail_is_caught(monkeypatch):
    orig = ol.select_moduli_one_limb

    def unseeded(L, heads=1):
        h = list(o.ONE_LIMB_HEADS[:min(heads, L)])
        return h + o.select_moduli(L - len(h))
    monkeypatch.setattr(ol, "select_moduli_one_limb", unseeded)
    A, B = _tiny(31, 3, 4, 5)
    with pytest.raises((ValueError, AssertionError)):
        o.dgemm_one_limb(A, B, 14, heads=5, check_definition=True)
    monkeypatch.setattr(ol, "select_moduli_one_limb", orig)
    o.dgemm_one_limb(A, B, 14, heads=5, check_definition=True)
