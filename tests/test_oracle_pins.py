"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every check here is independent of the oracle's own arithmetic: printed
values (tests/golden/paper_values.json), closed forms, brute force on tiny
inputs, exact rationals and invariants. None needs a GPU.
"""

import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as o


# ---------------------------------------------------------------- Sec. III

def test_e2m1_values_and_doubled_set(paper):
    assert list(o.E2M1_MAGNITUDES) == [float(v) for v in paper["e2m1_values"]]
    assert o.doubled_set() == paper["doubled_set"]
    # every E2M1 value doubled is an integer, and S is closed under negation
    S = o.doubled_set()
    assert all(-c in S for c in S)


def test_e2m1_codes_round_trip():
    # code -> value -> doubled limb -> code, for all 16 codes except -0
    for code in range(16):
        v = o.e2m1_decode(code)
        c = int(2 * v)
        assert 2 * v == c
        if code == 0x8:      # -0 encodes the same limb as +0
            assert o.e2m1_code(c) == 0
        else:
            assert o.e2m1_code(c) == code


def test_doubly_covered_classes(paper):
    S = o.doubled_set()
    counts = {r: sum(1 for c in S if c % 13 == r) for r in range(13)}
    assert all(v >= 1 for v in counts.values())          # Lemma 1: S covers Z/13
    assert sorted(r for r, v in counts.items() if v == 2) == paper["doubly_covered_classes_mod13"]


# ---------------------------------------------------------------- Lemma 1 / 2

def test_gap_free_range_values(paper):
    assert [o.gap_free_range(p) for p in (1, 2, 3)] == paper["gap_free_ranges"]


@pytest.mark.parametrize("p", [1, 2, 3, 4, 5])
def test_greedy_covers_exactly_gap_free_range(p):
    X = o.gap_free_range(p)
    for N in range(-X, X + 1):
        limbs = o.limb_decompose(N, p)
        assert sum(c * 13 ** i for i, c in enumerate(limbs)) == N
        assert all(abs(c) <= 8 for c in limbs)
    for N in (X + 1, -X - 1):
        with pytest.raises(ValueError):
            o.limb_decompose(N, p)


@pytest.mark.parametrize("p", [1, 2, 3, 4])
def test_any_digit_gap_free_range_brute_force(p):
    """Brute force over every p-limb combination: the largest gap-free
    interval around 0 is exactly X_p (Lemma 1)."""
    S = o.doubled_set()
    vals = {0}
    for _ in range(p):
        vals = {v * 13 + c for v in vals for c in S}
    X = 0
    while (X + 1) in vals and -(X + 1) in vals:
        X += 1
    assert X == o.gap_free_range(p)


def test_greedy_digit_properties(paper):
    S = set(o.doubled_set())
    for x in range(-500, 501):
        d = o.greedy_digit(x)
        assert d in S
        assert (x - d) % 13 == 0
        assert abs(d) <= paper["greedy_max_limb"]
        # smallest magnitude in the class, except the +-5 classes (Lemma 2)
        smallest = min((c for c in range(-6, 7) if (x - c) % 13 == 0), key=abs)
        if abs(smallest) != 5:
            assert d == smallest


def test_limb_counts(paper):
    lc = paper["limb_counts"]
    assert o.limbs_needed(128) == lc["int8"]
    assert o.limbs_needed(2 ** 24) == lc["fp32"]
    assert o.limbs_needed(2 ** 53) == lc["fp64"]
    assert o.limbs_needed(2 ** 53) ** 2 == paper["ozi_fp64_gemms"]
    assert o.limbs_needed(128) ** 2 == paper["int8_gemms"]


def test_lemma2_bounds(paper):
    assert (2 ** 24) // 144 == paper["lemma2_k_bound"]
    assert (2 ** 18) // 15 == paper["lemma2_greedy_group_bound"]
    # the deepest group of a 15 x 15 expansion has 15 pairs
    assert max(sum(1 for i in range(15) if 0 <= g - i < 15) for g in range(29)) == 15


# ---------------------------------------------------------------- Sec. V-A

def test_two_limb_moduli_exhaustive(paper):
    found = o.two_limb_moduli(400)
    assert found == list(range(2, 114)) + paper["two_limb_exceptions_above_113"]
    # independent check of the four exceptions: direct search for each class
    S = o.doubled_set()
    for m in paper["two_limb_exceptions_above_113"]:
        for r in range(m):
            assert any((c0 + 13 * c1 - r) % m == 0 for c0 in S for c1 in S)
    # and 114 fails (smallest-magnitude reasoning alone would not show it)
    assert not o.is_two_limb_modulus(114)


def test_select_moduli_matches_printed_list(paper):
    assert o.select_moduli(19) == paper["moduli_L19"]
    assert o.select_moduli(12) == paper["moduli_L19"][:12]
    m20 = o.select_moduli(20)
    assert m20[:19] == paper["moduli_L19"] and m20[19] == 47
    for a, b in itertools.combinations(m20, 2):
        assert math.gcd(a, b) == 1


def test_product_and_crt_condition(paper):
    P = o.moduli_product(paper["moduli_L19"])
    assert round(math.log2(P)) == paper["log2_P_approx"]
    assert 2 * 16384 * 2 ** 106 == 2 ** paper["crt_lhs_at_16384_log2"]
    assert 2 * 16384 * 2 ** 106 < P
    # L = 18 (prefix) fails Eq. (crt) at K = 16384
    assert o.moduli_product(paper["moduli_L19"][:18]) < 2 ** 121


def test_worked_example_115(paper):
    ex = paper["worked_example_115"]
    c0, c1 = o.two_limb_split(ex["class"], ex["m"])
    assert (c0, c1) == (ex["c0"], ex["c1"])
    assert c0 + 13 * c1 == ex["representative"]
    # and 57 itself is not two-limb representable by the greedy split
    with pytest.raises(ValueError):
        o.limb_decompose(57, 2)


def test_two_limb_round_trip_every_residue():
    """Every residue of every modulus (L = 20) -> canonical limbs -> E2M1 codes
    -> decoded values -> doubled limbs -> c0 + 13 c1 = r (mod m)."""
    for m in o.select_moduli(20):
        for r in range(m):
            c0, c1 = o.two_limb_split(r, m)
            v0 = o.e2m1_decode(o.e2m1_code(c0))
            v1 = o.e2m1_decode(o.e2m1_code(c1))
            d0, d1 = int(2 * v0), int(2 * v1)
            assert (d0, d1) == (c0, c1)
            assert (d0 + 13 * d1 - r) % m == 0
            assert abs(d0) <= 8 and abs(d1) <= 8        # +-12 never used


def test_karatsuba_moduli(paper):
    """Moduli whose every class has a two-limb split with the sum limb
    c0 + c1 also in S (Sec. V-A)."""
    S = set(o.doubled_set())

    def ok(m):
        return len({(c0 + 13 * c1) % m for c0 in S for c1 in S if c0 + c1 in S}) == m

    got = [m for m in paper["moduli_L19"] if ok(m)]
    assert got == paper["karatsuba_moduli"]
    assert o.karatsuba_moduli(paper["moduli_L19"]) == paper["karatsuba_moduli"]
    assert 4 * 19 - 1 - len(got) == paper["karatsuba_gemm_count"]
    assert 4 * 19 - 1 == paper["gemm_count_required"]
    assert 4 * 19 == paper["gemm_count_executed"]


def test_sum_limb_split_valid_symmetric_and_bounded():
    """Every residue of every Karatsuba modulus among the 20: the limbs and
    their sum are in S, within +-8, congruent to r; the split of -r is the
    negated split of r; where the canonical split already qualifies it is
    kept. With |c| <= 8 and one term per accumulator the FP32 bound of
    Lemma 3 holds up to the library's largest k."""
    S = set(o.doubled_set())
    kmods = o.karatsuba_moduli(o.select_moduli(20))
    assert kmods == [83, 73, 71, 67, 61, 59, 53, 47]
    changed = 0
    for m in kmods:
        for r in range(m):
            c0, c1 = o.sum_limb_split(r, m)
            assert (c0 + 13 * c1 - r) % m == 0
            for c in (c0, c1, c0 + c1):
                assert c in S and abs(c) <= 8
            n0, n1 = o.sum_limb_split((-r) % m, m)
            assert (n0, n1) == (-c0, -c1)
            k0, k1 = o.two_limb_split(r, m)
            if k0 + k1 in S and abs(k0 + k1) <= 8:
                assert (c0, c1) == (k0, k1)
            else:
                changed += 1
    assert changed > 0
    assert o.fp32_exact_bound(o.MAX_K_FP32, max_limb=8, terms=1)
    assert not o.fp32_exact_bound(o.MAX_K_FP32, max_limb=12, terms=1)


def test_karatsuba_residues_equal_exact_product():
    """r from the three Karatsuba products equals (A~ B~) mod m computed from
    the exact integer product, for every Karatsuba modulus."""
    rng = np.random.default_rng(11)
    Ai = rng.integers(-(1 << 40), 1 << 40, size=(9, 37), dtype=np.int64)
    Bi = rng.integers(-(1 << 40), 1 << 40, size=(37, 6), dtype=np.int64)
    exact = o.exact_int_matmul(Ai, Bi)
    for m in o.karatsuba_moduli(o.select_moduli(20)):
        got = o.residue_products_karatsuba(Ai, Bi, m)
        want = np.vectorize(lambda v: v % m, otypes=[object])(exact).astype(np.int64)
        assert np.array_equal(got["r"], want), m
        assert np.array_equal(got["r"], o.residue_products(Ai, Bi, m)["r"]), m
        a0, a1, as_ = o.limb_planes_karatsuba(Ai, m)
        assert np.array_equal(as_, a0 + a1)
        assert np.array_equal(np.mod(a0 + 13 * a1 - Ai, m), np.zeros_like(Ai))


def test_dgemm_karatsuba_route_identical():
    rng = np.random.default_rng(5)
    A = rng.standard_normal((7, 40))
    B = rng.standard_normal((40, 5))
    r1 = o.dgemm(A, B, 19, karatsuba=True, check_definition=True)
    r2 = o.dgemm(A, B, 19, karatsuba=False)
    assert np.array_equal(r1["C"].view(np.int64), r2["C"].view(np.int64))


def test_greedy_moduli_beyond_twenty_keep_the_rule():
    """The wide-range extension takes the next moduli of the same greedy rule
    (Sec. V-A): every pick is a two-limb modulus coprime to all earlier ones,
    and every skipped two-limb modulus between picks shares a factor with an
    earlier pick."""
    ms = o.select_moduli(27)
    assert ms[:19] == o.select_moduli(19)
    assert ms[19:] == [47, 43, 41, 31, 29, 19, 17, 11]
    two = set(o.two_limb_moduli())
    for i, m in enumerate(ms):
        assert m in two
        assert all(math.gcd(m, q) == 1 for q in ms[:i])
    for i in range(1, len(ms)):
        for skipped in range(ms[i] + 1, ms[i - 1]):
            if skipped in two:
                assert any(math.gcd(skipped, q) > 1 for q in ms[:i]), skipped
    # 42-bit CRT chunks stay exact: R (2^42 - 1) < 2^53 with R = sum (m - 1)
    assert sum(m - 1 for m in ms) * ((1 << 42) - 1) < (1 << 53)
    assert o.moduli_product(ms).bit_length() <= 4 * 42


def test_wide_capacity_closed_form():
    """c_A = min(cmax, ceil(b/2)), c_B = min(cmax, b - c_A) with b the largest
    integer such that 2 k 2^b < P; 23 moduli at k = 32768 give c = 63."""
    for L, k in ((23, 32768), (24, 131072), (21, 4096), (19, 32768)):
        ms = o.select_moduli(L)
        P = o.moduli_product(ms)
        for cmax in (53, 58, 63):
            cA, cB = o.capacity_bits(k, ms, cmax)
            b = max(bb for bb in range(400) if 2 * k * (1 << bb) < P)
            assert (cA, cB) == (min(cmax, (b + 1) // 2), min(cmax, b - min(cmax, (b + 1) // 2)))
            assert k * (1 << (cA + cB)) * 2 < P
    assert o.capacity_bits(32768, o.select_moduli(23), 63) == (63, 63)
    assert o.capacity_bits(32768, o.select_moduli(23)) == (53, 53)
    with pytest.raises(ValueError):
        o.capacity_bits(100, o.select_moduli(19), 64)


def test_wide_capacity_tiny_matrices_against_definition():
    """Brute force with c up to 63: the residue route equals the exact
    definition (Python-int sums of the converted operands, one rounding)."""
    rng = np.random.default_rng(17)
    for trial in range(6):
        m, n, k = 3, 4, 5 + trial
        A = (rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-40, 40, size=(m, k)))
        B = (rng.random((k, n)) - 0.5) * np.exp2(rng.integers(-40, 40, size=(k, n)))
        for L in (21, 23, 25):
            got = o.dgemm(A, B, L, cmax=63, check_definition=True)
            assert max(got["cA"], got["cB"]) > 53
            want = o.dgemm_definition(A, B, L, cmax=63)
            assert np.array_equal(got["C"].view(np.int64), want.view(np.int64))


def test_wide_capacity_is_more_accurate_at_phi_4():
    """With rows spanning many binades (phi = 4) the 53-bit cap truncates the
    small elements; 63 bits with 23 moduli cut the normalized error by at
    least 2^8 on a sample."""
    from paper_2608_06812_amd.workloads import dgemm_inputs
    A, B = dgemm_inputs(6, 6, 2048, 4.0, 404)
    e53 = e63 = 0.0
    c53 = o.dgemm(A, B, 19)["C"]
    c63 = o.dgemm(A, B, 23, cmax=63)["C"]
    for i in range(6):
        for j in range(6):
            e53 = max(e53, o.normalized_error(c53[i, j], A, B, i, j))
            e63 = max(e63, o.normalized_error(c63[i, j], A, B, i, j))
    assert e63 * 2 ** 8 <= e53
    assert e63 < 2.0 ** -40


def test_best_18_set_below_printed_bound(paper):
    """Branch and bound over pairwise-coprime 18-subsets of the two-limb
    moduli: the best product is below 2^117.80 and below 2^121, so L = 19 is
    minimal (Sec. V-A)."""
    cands = sorted(o.two_limb_moduli(400), reverse=True)
    logs = [math.log2(m) for m in cands]
    best = [0.0]

    def rec(start, chosen, total):
        if len(chosen) == 18:
            best[0] = max(best[0], total)
            return
        need = 18 - len(chosen)
        for i in range(start, len(cands)):
            if len(cands) - i < need:
                return
            # optimistic bound: the next `need` candidates, ignoring coprimality
            if total + sum(logs[i:i + need]) <= best[0]:
                return
            m = cands[i]
            if all(math.gcd(m, q) == 1 for q in chosen):
                chosen.append(m)
                rec(i + 1, chosen, total + logs[i])
                chosen.pop()

    rec(0, [], 0.0)
    assert best[0] <= paper["best_18_set_log2_at_most"] + 5e-3
    assert best[0] > paper["best_18_set_log2_at_most"] - 5e-3
    assert best[0] < 121


# ---------------------------------------------------------------- Lemma 3

def test_lemma3_bounds(paper):
    b = paper["lemma3_bounds"]
    assert (2 ** 24) // 144 == b["partial_product"]
    assert (2 ** 24) // 288 == b["cross_term"]
    factor = (1 + 2 * 13 + 169) * 144
    assert factor == paper["lemma3_composition_factor"]
    assert (2 ** 31) // factor == b["composition_int32"]
    P = o.moduli_product(paper["moduli_L19"])
    kmax = max(K for K in range(76000, 77000) if 2 * K * 2 ** 106 < P)
    assert kmax == b["crt"]


def test_fp32_exactness_proof():
    """Worst-case partial sums of the limb products fit FP32 exactly up to
    K = 131,072 with greedy limbs (|c| <= 8, two terms in the cross-term
    accumulator), and no further."""
    assert o.fp32_exact_bound(o.MAX_K_FP32, max_limb=8, terms=2)
    assert not o.fp32_exact_bound(o.MAX_K_FP32 + 1, max_limb=8, terms=2)
    # the paper's bound with |c| <= 12 (Lemma 3, cross term)
    assert o.fp32_exact_bound(58254, max_limb=12, terms=2)
    assert not o.fp32_exact_bound(58255, max_limb=12, terms=2)


@pytest.mark.slow
def test_fp32_accumulation_emulated_adversarial():
    """Sequential FP32 accumulation of an adversarial cross-term (all limbs 8
    except a final 1 x 1 product that only the last quarter bit carries)
    equals the integer sum at K = 131,072; a longer sum past the bound loses
    that quarter."""
    K = o.MAX_K_FP32
    a = np.full(2 * K, 8, dtype=np.int64)
    b = np.full(2 * K, 8, dtype=np.int64)
    a[-1] = b[-1] = 1
    a[-2] = b[-2] = 0                  # keep the total just below the bound
    exact = int(np.dot(a, b))
    assert o.fp32_accumulate_emulated(a, b) == exact
    a2 = np.concatenate([np.full(64, 8), a])
    b2 = np.concatenate([np.full(64, 8), b])
    assert o.fp32_accumulate_emulated(a2, b2) != int(np.dot(a2, b2))


# ---------------------------------------------------------------- Sec. V-B

def test_crt_weights_are_idempotents():
    mods = o.select_moduli(20)
    for L in (2, 14, 19, 20):
        ms = mods[:L]
        w = o.crt_weights(ms)
        for i, wi in enumerate(w):
            for j, mj in enumerate(ms):
                assert wi % mj == (1 if i == j else 0)


def test_crt_footnote_constants(paper):
    ms = paper["moduli_L19"]
    P = o.moduli_product(ms)
    w = o.crt_weights(ms)
    assert sum(m - 1 for m in ms) == paper["crt_quotient_bound"]
    Smax = sum((m - 1) * wi for m, wi in zip(ms, w))
    assert Smax // P == paper["crt_quotient_max"]
    assert Smax < 2 ** paper["crt_sum_log2_below"]


def test_crt_round_trip_random_integers():
    rng = np.random.default_rng(7)
    for L in (3, 14, 19, 20):
        ms = o.select_moduli(L)
        P = o.moduli_product(ms)
        xs = [int(rng.integers(-2 ** 62, 2 ** 62)) * int(rng.integers(1, 2 ** 40)) % P - P // 2
              for _ in range(64)]
        xs += [0, 1, -1, (P - 1) // 2, -((P - 1) // 2)]
        res = [np.array([x % m for x in xs], dtype=np.int64) for m in ms]
        back = o.crt_reconstruct(res, ms)
        assert list(back) == xs
        for idx, x in enumerate(xs):
            assert o.crt_reconstruct_paper([int(r[idx]) for r in res], ms) == x


# ---------------------------------------------------------------- Sec. IV-B

def test_floor_log2_against_exact():
    vals = [1.0, 2.0, 3.0, 0.75, 1e-300, 5e-324, 2.2250738585072014e-308,
            1.7976931348623157e308, 1.5 * 2 ** -1060, 123456.789]
    for v in vals:
        e = o.floor_log2(v)
        f = Fraction(v)
        assert Fraction(2) ** e <= f < Fraction(2) ** (e + 1)


def test_to_integers_vectorised_matches_exact_rounding():
    rng = np.random.default_rng(3)
    X = np.array([[2.5, 3.5, -2.5, -0.5, 0.5, 1.5, 5e-324, -1e-310],
                  [1e300, 3e299, -1e-300, 7.0, 0.0, -0.0, 2.0 ** 52 + 1, 1.0]])
    X = np.concatenate([X, rng.standard_normal((3, 8)) * np.exp(8 * rng.standard_normal((3, 8)))])
    for c in (53, 42, 20, 3):
        s = o.shift_exponents(X, axis=1, c=c)
        a = o.to_integers(X, s, axis=1)
        b = o.to_integers_fraction(X, s, axis=1)
        assert np.array_equal(a, b)
        assert np.all(np.abs(a) <= 2 ** c)
        # row maxima convert to [2^(c-1), 2^c]
        mx = np.max(np.abs(a), axis=1)
        assert np.all((mx >= 2 ** (c - 1)) & (mx <= 2 ** c))
    # ties round to even
    s = np.zeros(1, dtype=np.int64)
    got = o.to_integers_fraction(np.array([[0.5, 1.5, 2.5, -0.5, -1.5]]), s, axis=1)
    assert list(got[0]) == [0, 2, 2, 0, -2]


def test_zero_row_and_column_shift_zero():
    X = np.array([[0.0, 0.0], [1.0, 0.0]])
    assert list(o.shift_exponents(X, axis=1, c=53)) == [0, 52]
    assert list(o.shift_exponents(X, axis=0, c=53)) == [52, 0]


def test_capacity_rule():
    m19 = o.select_moduli(19)
    # the paper's setting: c = 53 for L = 19 and K <= 76,549
    assert o.capacity_bits(16384, m19) == (53, 53)
    assert o.capacity_bits(76549, m19) == (53, 53)
    for L in range(2, 21):
        ms = o.select_moduli(L)
        P = o.moduli_product(ms)
        for k in (1, 7, 256, 4096, 16384, 32768):
            try:
                cA, cB = o.capacity_bits(k, ms)
            except ValueError:
                assert 2 * k * 2 ** 2 >= P
                continue
            assert 2 * k * 2 ** (cA + cB) < P
            assert 1 <= cB <= cA <= 53
            if cA < 53 and cB < 53:
                assert 2 * k * 2 ** (cA + cB + 1) >= P     # as large as allowed


def test_round_scaled_special_cases():
    tiny = 2.0 ** -1074
    assert o.round_scaled(3, 1076) == tiny            # 0.75 ulp -> 1 ulp
    assert o.round_scaled(1, 1075) == 0.0             # half ulp, tie to even 0
    assert o.round_scaled(3, 1075) == 2 * tiny        # 1.5 ulp -> 2 (even)
    assert o.round_scaled(5, 1075) == 2 * tiny        # 2.5 ulp -> 2 (even)
    assert o.round_scaled(-3, 1076) == -tiny
    assert o.round_scaled(2 ** 53 + 1, 0) == 2.0 ** 53          # tie to even
    assert o.round_scaled(2 ** 53 + 3, 0) == 2.0 ** 53 + 4
    assert o.round_scaled(1, -1024) == math.inf
    assert o.round_scaled(-1, -1024) == -math.inf
    assert o.round_scaled(2 ** 53 - 1, -971) == 1.7976931348623157e308
    assert o.round_scaled(2 ** 54 - 1, -970) == math.inf    # rounds up past the max
    assert o.round_scaled(0, 5) == 0.0 and math.copysign(1, o.round_scaled(0, 5)) == 1
    rng = np.random.default_rng(11)
    for _ in range(200):
        x = int(rng.integers(-2 ** 53, 2 ** 53))
        sh = int(rng.integers(-900, 900))
        assert o.round_scaled(x, sh) == math.ldexp(float(x), -sh)   # exact cases


# ---------------------------------------------------------------- whole method

def _binade_matrix(rng, shape, spread):
    X = (rng.random(shape) - 0.5) * np.exp2(rng.integers(-spread, spread + 1, size=shape))
    X[rng.random(shape) < 0.1] = 0.0
    return X


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_tiny_matrices(seed):
    """Tiny matrices through the residue route vs the exact integer
    definition of the result (Python ints, no residues)."""
    rng = np.random.default_rng(100 + seed)
    m, n, k = (int(v) for v in rng.integers(1, 7, size=3))
    A = _binade_matrix(rng, (m, k), 40)
    B = _binade_matrix(rng, (k, n), 40)
    if seed == 0:
        A[0, :] = 0.0                       # zero row
        B[:, -1] = 0.0                      # zero column
    if seed == 1:
        A[-1, 0] = 5e-324                   # subnormal entries
        B[0, 0] = -3e-320
    for L in (3, 8, 14, 19):
        try:
            res = o.dgemm(A, B, L, check_definition=True)
        except ValueError:
            assert L == 3
            continue
        assert np.array_equal(res["C"], o.dgemm_definition(A, B, L))


def test_phi0_paper_law_is_correctly_rounded_product():
    """With the paper's law at phi = 0 every entry is +-(1+u), the conversion
    is exact (c = 53), and C must equal fl(AB) bit for bit (Sec. VII-A)."""
    rng = np.random.default_rng(5)
    m, n, k = 6, 5, 64
    A = rng.choice([-1.0, 1.0], size=(m, k)) * (1 + rng.random((m, k)))
    B = rng.choice([-1.0, 1.0], size=(k, n)) * (1 + rng.random((k, n)))
    C = o.dgemm(A, B, 19)["C"]
    for i in range(m):
        for j in range(n):
            assert C[i, j] == float(o.exact_product_entry(A, B, i, j))


@pytest.mark.slow
def test_accuracy_against_printed_bits(paper):
    """Paper law at phi = 0 and 32, K = 8192, L = 19: the normalized error of
    a 4 x 4 sample is in line with the printed maxima over 128 x 128
    (58.2 and 52.3 bits); a sample's maximum can only be smaller."""
    K = 8192
    for phi, printed in ((0, paper["accuracy_bits_phi0"]), (32, paper["accuracy_bits_phi32"])):
        rng = np.random.default_rng(20260806 + phi)
        A = rng.choice([-1.0, 1.0], size=(4, K)) * (1 + rng.random((4, K))) * np.exp2(rng.integers(0, phi + 1, size=(4, K)))
        B = rng.choice([-1.0, 1.0], size=(K, 4)) * (1 + rng.random((K, 4))) * np.exp2(rng.integers(0, phi + 1, size=(K, 4)))
        C = o.dgemm(A, B, 19)["C"]
        worst = max(o.normalized_error(C[i, j], A, B, i, j) for i in range(4) for j in range(4))
        bits = -math.log2(worst) if worst > 0 else 99
        assert printed - 1.0 <= bits <= printed + 4.0, (phi, bits)


@pytest.mark.slow
def test_config1_full_oracle_definition():
    """256^3 with the (U - 0.5) exp(0.5 N) law and 14 moduli: the residue
    route equals the exact integer product for every entry."""
    from paper_2608_06812_amd.workloads import dgemm_inputs
    A, B = dgemm_inputs(256, 256, 256, phi=0.5, seed=20260806)
    res = o.dgemm(A, B, 14, check_definition=True)
    assert (res["cA"], res["cB"]) == (42, 42)
    assert np.all(np.isfinite(res["C"]))


# ---------------------------------------------------------------- Sec. III (INT8)

def test_int8_limbs_cover_every_int8():
    for v in range(-128, 128):
        limbs = o.limb_decompose(v, 3)
        assert sum(c * 13 ** i for i, c in enumerate(limbs)) == v
        assert all(abs(c) <= 8 for c in limbs)


@pytest.mark.parametrize("seed", range(3))
def test_int8_limb_route_equals_integer_product(seed):
    rng = np.random.default_rng(seed)
    m, n, k = 9, 7, 300
    A = rng.integers(-128, 128, size=(m, k)).astype(np.int8)
    B = rng.integers(-128, 128, size=(k, n)).astype(np.int8)
    if seed == 0:
        A[0, :] = -128
        B[:, 0] = -128
    ref = (A.astype(object) @ B.astype(object))
    got = o.igemm_s8(A, B)
    assert np.array_equal(got.astype(np.int64), ref.astype(np.int64))
    assert np.array_equal(o.igemm_s8_limbs(A, B), got)


def test_int8_wraps_like_int32():
    A = np.full((1, 140000), -128, dtype=np.int8)
    B = np.full((140000, 1), -128, dtype=np.int8)
    exact = 128 * 128 * 140000
    assert exact >= 2 ** 31
    assert int(o.igemm_s8(A, B)[0, 0]) == exact - 2 ** 32


# ---------------------------------------------------------------- exact block products

@pytest.mark.parametrize("seed", range(4))
def test_exact_block_matches_fraction_sums(seed):
    """The digit-split exact block product equals plain Fraction sums,
    including zeros, subnormals and large exponent spreads."""
    rng = np.random.default_rng(40 + seed)
    m, n, k = 5, 4, 37
    A = (rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-60, 60, size=(m, k)))
    B = (rng.random((k, n)) - 0.5) * np.exp2(rng.integers(-60, 60, size=(k, n)))
    A[rng.random((m, k)) < 0.2] = 0.0
    A[0, 0] = 5e-324
    B[1, 1] = -2.5e-310
    if seed == 1:
        A[2, :] = 0.0
    rows, cols = [0, 2, 4], [1, 3]
    P, S = o.exact_block(A, B, rows, cols)
    for a, i in enumerate(rows):
        for b, j in enumerate(cols):
            assert P[a, b] == o.exact_product_entry(A, B, i, j)
            want = sum((abs(Fraction(float(A[i, q]))) * abs(Fraction(float(B[q, j]))) for q in range(k)),
                       Fraction(0))
            assert S[a, b] == want


def test_normalized_errors_block_matches_single_entry():
    rng = np.random.default_rng(9)
    A = rng.standard_normal((3, 50))
    B = rng.standard_normal((50, 3))
    C = A @ B
    got = o.normalized_errors_block(C, A, B, range(3), range(3))
    for i in range(3):
        for j in range(3):
            assert got[i, j] == o.normalized_error(C[i, j], A, B, i, j)


# ---------------------------------------------------------------- Sec. IV-B error bound

@pytest.mark.parametrize("phi,seed", [(4.0, 1), (8.0, 2), (0.5, 3)])
def test_quantization_bound_holds_exactly(phi, seed):
    """|C - AB| against the exact product stays within the a-priori bound of
    the shared-exponent conversion on every element (wide exponent spread)."""
    from paper_2608_06812_amd.workloads import dgemm_inputs
    A, B = dgemm_inputs(12, 10, 300, phi, seed)
    res = o.dgemm(A, B, 19)
    rows, cols = np.arange(12), np.arange(10)
    bound = o.quantization_error_bound(A, B, res["s"], res["t"], res["x"], rows, cols)
    exact, _ = o.exact_block(A, B, rows, cols)
    for i in range(12):
        for j in range(10):
            err = abs(Fraction(float(res["C"][i, j])) - exact[i, j])
            assert err <= Fraction(float(bound[i, j]))


def test_quantization_bound_is_attained_by_a_half_unit_loss():
    """A row whose small element sits exactly half a unit of the row's
    scale below an integer loses exactly that half unit (ties to even):
    the bound's A term is reached up to the other terms."""
    k = 4
    A = np.array([[1.0, 2.0 ** -53, 0.0, 0.0]])          # s = 52: 2^-53 -> 0.5 -> rounds to 0
    B = np.array([[0.0], [1.0], [0.0], [0.0]])
    res = o.dgemm(A, B, 19)
    assert int(res["s"][0]) == 52 and int(res["Ai"][0, 1]) == 0
    err = abs(float(res["C"][0, 0]) - 2.0 ** -53)
    bound = o.quantization_error_bound(A, B, res["s"], res["t"], res["x"], [0], [0])[0, 0]
    assert err == 2.0 ** -53 and err <= bound <= 4 * err
