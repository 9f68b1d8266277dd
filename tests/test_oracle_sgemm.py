"""Pins of the FP32-emulation oracle (oracle/sgemm_fp4.py): the binary32
rounding against numpy's single rounding of exact doubles and against
hand-derived special cases (ties, subnormal boundaries, overflow, and a
value where rounding first to FP64 would give the wrong FP32), the capacity
rule against a brute-force search, the residue route against the exact
definition, and correctly rounded results on exactly convertible inputs."""

import random
from fractions import Fraction

import numpy as np
import pytest

import oracle as o
from paper_2608_06812_amd.workloads import dgemm_inputs, paper_law_inputs


def _f32(v):
    return np.float32(v)


def test_round_scaled_f32_matches_numpy_on_exact_doubles():
    """x < 2^53 and results in the normal FP64 range: x 2^-shift is an
    exact double, so numpy's float64 -> float32 cast is a single rounding."""
    rng = random.Random(3)
    for _ in range(20000):
        x = rng.randint(-(1 << 53) + 1, (1 << 53) - 1)
        sh = rng.randint(-150, 320)
        with np.errstate(over="ignore"):
            want = np.float32(np.ldexp(np.float64(x), -sh))
        got = o.round_scaled_f32(x, sh)
        assert got.view(np.uint32) == want.view(np.uint32), (x, sh)


def test_round_scaled_f32_special_cases():
    two = Fraction(2)
    tiny = np.float32(2.0 ** -149)
    assert o.round_scaled_f32(1, 149) == tiny
    assert o.round_scaled_f32(1, 150) == 0.0                  # tie to even (zero)
    assert o.round_scaled_f32(3, 151) == tiny                 # 0.75 ulp -> 1 ulp
    assert o.round_scaled_f32(3, 150) == np.float32(2.0 ** -148)   # 1.5 ulp tie -> 2 ulp
    assert o.round_scaled_f32(-1, 151).view(np.uint32) == np.float32(-0.0).view(np.uint32)
    assert o.round_scaled_f32(1 << 23, 149 + 23) == tiny
    fmax = (2 ** 24 - 1) * 2 ** 104
    assert o.round_scaled_f32(fmax, 0) == np.finfo(np.float32).max
    assert o.round_scaled_f32(2 * fmax + 2 ** 104, 1) == np.inf      # tie above max -> inf
    assert o.round_scaled_f32(2 * fmax + 2 ** 104 - 1, 1) == np.finfo(np.float32).max
    assert o.round_scaled_f32(-(1 << 200), 0) == -np.inf
    # 2^24 + 1 + 2^-30: rounding first to FP64 gives 2^24 + 1, a tie, and
    # then 2^24; the single rounding gives 2^24 + 2
    x = ((2 ** 24 + 1) << 30) + 1
    assert o.round_scaled_f32(x, 30) == np.float32(2 ** 24 + 2)
    assert float(Fraction(x) / two ** 30) == 2 ** 24 + 1


@pytest.mark.parametrize("L", [2, 5, 9, 10, 12, 19])
def test_capacity_fp32_brute_force(L):
    moduli = o.select_moduli(L)
    P = o.moduli_product(moduli)
    for k in (1, 7, 256, 16384, 131072):
        b = 0
        while 2 * k * 2 ** (b + 1) < P:
            b += 1
        if b < 2:
            with pytest.raises(ValueError):
                o.capacity_bits_fp32(k, moduli)
            continue
        cA, cB = o.capacity_bits_fp32(k, moduli)
        assert cA + cB <= b and max(cA, cB) <= 24 and abs(cA - cB) <= 1
        assert cA + cB == min(b, 48)


def test_ten_moduli_give_fp32_capacity_at_16384():
    assert o.capacity_bits_fp32(16384, o.select_moduli(10)) == (24, 24)
    assert o.capacity_bits_fp32(16384, o.select_moduli(9)) != (24, 24)


def test_sgemm_residue_route_equals_definition():
    rng = np.random.default_rng(21)
    for L in (6, 10, 14):
        for _ in range(3):
            m, n, k = 3, 4, 6
            A = ((rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-40, 40, size=(m, k)))).astype(np.float32)
            B = ((rng.random((k, n)) - 0.5) * np.exp2(rng.integers(-40, 40, size=(k, n)))).astype(np.float32)
            got = o.sgemm(A, B, L)
            assert got["C"].dtype == np.float32
            assert np.array_equal(got["C"].view(np.uint32), o.sgemm_definition(A, B, L).view(np.uint32))
            assert np.all(got["x"] == o.exact_int_matmul(got["Ai"], got["Bi"]))


def test_sgemm_exactly_convertible_is_correctly_rounded():
    """FP32 entries in [1, 2) (phi = 0 of the paper's law, cast to FP32):
    conversion with c = 24 is exact, so C is RN32 of the exact product."""
    A, B = paper_law_inputs(5, 6, 40, 0, 9)
    A, B = A.astype(np.float32), B.astype(np.float32)
    res = o.sgemm(A, B, 10)
    assert (res["cA"], res["cB"]) == (24, 24)
    for i in range(5):
        for j in range(6):
            exact = o.exact_product_entry(A.astype(np.float64), B.astype(np.float64), i, j)
            want = o.round_scaled_f32(exact.numerator, 0) if exact.denominator == 1 else \
                o.round_scaled_f32(exact.numerator * (2 ** 60 // exact.denominator), 60)
            assert res["C"][i, j] == want


def test_sgemm_accuracy_band():
    """Normalized error within a few FP32 units (2^-22) on the phi = 0.5
    law, no worse than a plain FP32-accumulated product's."""
    A, B = dgemm_inputs(24, 24, 512, 0.5, 17)
    A, B = A.astype(np.float32), B.astype(np.float32)
    C = o.sgemm(A, B, 10)["C"]
    A64, B64 = A.astype(np.float64), B.astype(np.float64)
    err = o.normalized_errors_block(C.astype(np.float64), A64, B64, np.arange(24), np.arange(24))
    assert err.max() <= 2.0 ** -22
    native = (A @ B).astype(np.float64)
    err_n = o.normalized_errors_block(native, A64, B64, np.arange(24), np.arange(24))
    assert err.max() <= max(err_n.max(), 2.0 ** -23)
