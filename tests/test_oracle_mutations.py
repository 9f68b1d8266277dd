"""Plant plausible mistakes in the oracle (CPU only) and check that the pins
catch each one: a dropped term, a wrong weight, a sign slip, a transposed
operand, a wrong rounding mode."""

import numpy as np
import pytest

import oracle as o
from oracle import ozaki2_fp4 as mod


_ROUTE = {"karatsuba": False}


def _tiny_mismatch():
    """True when the residue route disagrees with the exact definition on a
    few tiny matrices (the brute-force pin), or raises an internal check."""
    rng = np.random.default_rng(1)
    for _ in range(4):
        m, n, k = 3, 4, 5
        A = (rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-30, 30, size=(m, k)))
        B = (rng.random((k, n)) - 0.5) * np.exp2(rng.integers(-30, 30, size=(k, n)))
        try:
            got = o.dgemm(A, B, 14, karatsuba=_ROUTE["karatsuba"])["C"]
        except (AssertionError, ValueError):
            return True
        if not np.array_equal(got, o.dgemm_definition(A, B, 14)):
            return True
    return False


def _round_trip_fails():
    try:
        for m in o.select_moduli(20):
            for r in range(m):
                c0, c1 = o.two_limb_split(r, m)
                d0 = int(2 * o.e2m1_decode(o.e2m1_code(c0)))
                d1 = int(2 * o.e2m1_decode(o.e2m1_code(c1)))
                if (d0 + 13 * d1 - r) % m or abs(d0) > 8 or abs(d1) > 8:
                    return True
    except (ValueError, KeyError):
        return True
    return False


def test_unmutated_oracle_passes():
    assert not _tiny_mismatch()
    assert not _round_trip_fails()


def test_wrong_composition_weight_is_caught(monkeypatch):
    orig = mod.residue_products

    def bad(Ai, Bi, m):
        out = orig(Ai, Bi, m)
        out["r"] = np.mod(out["G0"] + 169 * out["G1"] + 13 * out["G2"], m)   # weights swapped
        return out
    monkeypatch.setattr(mod, "residue_products", bad)
    assert _tiny_mismatch()


def test_dropped_cross_term_is_caught(monkeypatch):
    def bad(Ai, Bi, m):
        a0, a1 = o.limb_planes(Ai, m)
        b0, b1 = o.limb_planes(Bi, m)
        G0 = a0 @ b0
        G1 = a0 @ b1                       # a1 b0 dropped
        G2 = a1 @ b1
        return {"G0": G0, "G1": G1, "G2": G2, "r": np.mod(G0 + 13 * G1 + 169 * G2, m)}
    monkeypatch.setattr(mod, "residue_products", bad)
    assert _tiny_mismatch()


def test_transposed_operand_is_caught(monkeypatch):
    def bad(Ai, Bi, m):
        a0, a1 = o.limb_planes(Ai, m)
        b0, b1 = o.limb_planes(Bi, m)
        G0 = a0 @ b0
        G1 = a0 @ b1 + (b0.T @ a1.T).T[:, ::-1]     # wrong operand orientation
        G2 = a1 @ b1
        return {"G0": G0, "G1": G1, "G2": G2, "r": np.mod(G0 + 13 * G1 + 169 * G2, m)}
    monkeypatch.setattr(mod, "residue_products", bad)
    assert _tiny_mismatch()


def test_missing_symmetric_map_is_caught(monkeypatch):
    def bad(res, moduli):
        P = o.moduli_product(moduli)
        w = o.crt_weights(moduli)
        S = sum(np.asarray(r, dtype=np.int64).astype(object) * wi for r, wi in zip(res, w))
        return np.vectorize(lambda v: v % P, otypes=[object])(S)      # no x - P
    monkeypatch.setattr(mod, "crt_reconstruct", bad)
    assert _tiny_mismatch()


def test_greedy_without_replacement_is_caught(monkeypatch):
    monkeypatch.setattr(mod, "greedy_digit", lambda x: (x + 6) % 13 - 6)   # emits +-5
    assert _round_trip_fails()


def test_truncating_conversion_is_caught(monkeypatch):
    def bad(X, shifts, axis):
        sh = shifts[:, None] if axis == 1 else shifts[None, :]
        return np.trunc(np.ldexp(X, sh.astype(np.int64))).astype(np.int64)
    monkeypatch.setattr(mod, "to_integers", bad)
    # the conversion pin compares against exact half-to-even rounding
    X = np.array([[2.5, -3.7, 1e-3, 0.3]])
    s = o.shift_exponents(X, axis=1, c=3)
    assert not np.array_equal(mod.to_integers(X, s, axis=1), o.to_integers_fraction(X, s, axis=1))


def test_off_by_one_exponent_is_caught(monkeypatch):
    monkeypatch.setattr(mod, "floor_log2", lambda x: int(np.frexp(abs(x))[1]))   # e instead of e-1
    X = np.array([[3.0, 1.0]])
    # shift must take the row maximum into [2^(c-1), 2^c)
    s = o.shift_exponents(X, axis=1, c=10)
    v = o.to_integers(X, s, axis=1)
    assert not (2 ** 9 <= np.max(np.abs(v)) <= 2 ** 10)


def test_wrong_modulus_order_is_caught(monkeypatch, paper):
    monkeypatch.setattr(mod, "select_moduli", lambda L: sorted(o.two_limb_moduli())[:L])
    assert mod.select_moduli(19) != paper["moduli_L19"]


@pytest.mark.parametrize("bad_code", [{6: 6, 8: 5}, {1: 2, 2: 1}])
def test_wrong_e2m1_code_table_is_caught(monkeypatch, bad_code):
    table = dict(mod._CODE_OF_MAG)
    table.update(bad_code)
    monkeypatch.setattr(mod, "_CODE_OF_MAG", table)
    bad = False
    for c in o.doubled_set():
        if int(2 * o.e2m1_decode(o.e2m1_code(c))) != c:
            bad = True
    assert bad


def test_karatsuba_cross_term_without_p2_is_caught(monkeypatch):
    orig = mod.residue_products_karatsuba

    def bad(Ai, Bi, m):
        out = orig(Ai, Bi, m)
        out["r"] = np.mod(out["P0"] + 13 * (out["Ps"] - out["P0"]) + 169 * out["P2"], m)
        return out
    monkeypatch.setattr(mod, "residue_products_karatsuba", bad)
    monkeypatch.setitem(_ROUTE, "karatsuba", True)
    assert _tiny_mismatch()


def test_karatsuba_wrong_sum_plane_is_caught(monkeypatch):
    orig = mod.limb_planes_karatsuba

    def bad(Xi, m):
        c0, c1, _ = orig(Xi, m)
        return c0, c1, c0 - c1
    monkeypatch.setattr(mod, "limb_planes_karatsuba", bad)
    monkeypatch.setitem(_ROUTE, "karatsuba", True)
    assert _tiny_mismatch()


# ---------------------------------------------------------------- scheme I

from oracle import ozaki1_fp4 as mod1  # noqa: E402


def _ozi_mismatch():
    """True when the scheme-I oracle breaks one of its pins on small inputs:
    limbs outside S, the expansion differing from the integer product, or C
    differing from scheme II's (both at c = 53)."""
    S = set(o.doubled_set())
    rng = np.random.default_rng(2)
    for _ in range(3):
        m, n, k = 4, 3, 9
        A = (rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-20, 20, size=(m, k)))
        B = (rng.random((k, n)) - 0.5) * np.exp2(rng.integers(-20, 20, size=(k, n)))
        try:
            res = o.dgemm_ozi(A, B, 15)
        except (AssertionError, ValueError):
            return True
        if any(not set(np.unique(a).tolist()) <= S for a in res["a"] + res["b"]):
            return True
        if not np.all(res["x"] == o.exact_int_matmul(res["Ai"], res["Bi"])):
            return True
        if not np.array_equal(res["C"], o.dgemm(A, B, 18)["C"]):
            return True
    return False


def test_unmutated_scheme1_passes():
    assert not _ozi_mismatch()


def test_scheme1_wrong_group_weight_is_caught(monkeypatch):
    def bad(G):
        x = np.zeros(G[0].shape, dtype=object)
        for g, Gg in enumerate(G):
            x = x + Gg.astype(object) * (13 ** (g + (1 if g == len(G) - 1 else 0)))
        return x
    monkeypatch.setattr(mod1, "ozi_compose", bad)
    assert _ozi_mismatch()


def test_scheme1_off_by_one_group_is_caught(monkeypatch):
    def bad(a, b):
        p, q = len(a), len(b)
        G = []
        for g in range(p + q - 1):
            acc = np.zeros((a[0].shape[0], b[0].shape[1]), dtype=np.int64)
            for i in range(p):
                j = g - i + 1            # shifted anti-diagonal
                if 0 <= j < q:
                    acc = acc + mod._limb_matmul(a[i], b[j])
            G.append(acc)
        return G
    monkeypatch.setattr(mod1, "ozi_group_products", bad)
    assert _ozi_mismatch()


def test_scheme1_missing_minus5_substitution_is_caught(monkeypatch):
    def bad(Xi, p):
        rest = np.asarray(Xi, dtype=np.int64).copy()
        out = []
        for _ in range(p):
            c = np.mod(rest + 6, 13) - 6          # +-5 kept: not in S
            out.append(c)
            rest = (rest - c) // 13
        return out
    monkeypatch.setattr(mod1, "ozi_limbs", bad)
    assert _ozi_mismatch()


# ---------------------------------------------------------------- FP32 emulation

from fractions import Fraction  # noqa: E402

from oracle import sgemm_fp4 as mod32  # noqa: E402


def _f32_mismatch():
    """True when the FP32-emulation oracle breaks a pin: the single binary32
    rounding (a double-rounding case, a tie at the subnormal end) or the
    residue route against the exact definition."""
    x = ((2 ** 24 + 1) << 30) + 1
    if o.round_scaled_f32(x, 30) != np.float32(2 ** 24 + 2):
        return True
    if o.round_scaled_f32(3, 150) != np.float32(2.0 ** -148):
        return True
    rng = np.random.default_rng(5)
    A = ((rng.random((3, 5)) - 0.5) * np.exp2(rng.integers(-30, 30, size=(3, 5)))).astype(np.float32)
    B = ((rng.random((5, 2)) - 0.5) * np.exp2(rng.integers(-30, 30, size=(5, 2)))).astype(np.float32)
    try:
        got = o.sgemm(A, B, 10)["C"]
    except (AssertionError, ValueError):
        return True
    return not np.array_equal(got.view(np.uint32), o.sgemm_definition(A, B, 10).view(np.uint32))


def test_unmutated_fp32_passes():
    assert not _f32_mismatch()


def test_fp32_double_rounding_is_caught(monkeypatch):
    def bad(x, shift):
        return np.float32(float(Fraction(int(x)) / Fraction(2) ** int(shift)))
    monkeypatch.setattr(mod32, "round_scaled_f32", bad)
    monkeypatch.setattr(o, "round_scaled_f32", bad)
    assert _f32_mismatch()


def test_fp32_capacity_53_is_caught(monkeypatch):
    monkeypatch.setattr(mod32, "FP32_CAPACITY", 53)
    assert _f32_mismatch() or o.capacity_bits_fp32(16384, o.select_moduli(10)) != (24, 24)
