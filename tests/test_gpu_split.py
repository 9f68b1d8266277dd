"""GPU parity of the two-term split route (ozfp4_dgemm_split) against the
oracle (oracle/split2_fp4.py): C bit for bit on ragged shapes with wide
exponent spreads and several moduli counts (few moduli give small
capacities, so the second terms carry many bits), on shapes whose tile grid
takes the XCD-share mapping, on edge values (zero lines, subnormal inputs
and results, overflow to infinity, cancellation), at the largest k, and on
sampled outputs of the wide-dynamic-range workload (m = n = 8192,
k = 32768, phi = 4), where the normalized error must come within the final
rounding. Where every element lies within c + d bits of its line's largest
one (the paper's input law at phi = 32), C must be the correctly rounded
product fl(AB) in every element."""

import math

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, bits_equal, dev_cm, to_np
from paper_2608_06812_amd.workloads import dgemm_inputs, paper_law_inputs

pytestmark = pytest.mark.gpu

SEED = 20261301


def _wide(m, k, spread, seed):
    rng = np.random.default_rng(seed)
    X = (rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-spread, spread + 1, (m, k)))
    X[rng.random((m, k)) < 0.05] = 0.0
    return X


@pytest.mark.parametrize("m,n,k,L,spread", [
    (1, 1, 1, 19, 0), (131, 67, 129, 19, 40), (64, 80, 300, 4, 30), (33, 97, 64, 6, 200),
    (200, 130, 333, 12, 60), (300, 300, 200, 19, 100), (97, 31, 1000, 20, 10),
    (256, 256, 256, 27, 300)])
def test_split_bit_exact(gpu_lib, m, n, k, L, spread):
    A, B = _wide(m, k, spread, SEED + m), _wide(k, n, spread, SEED + n + 1)
    want = o.dgemm_split2(A, B, L)["C"]
    announce(f"dgemm_split m={m} n={n} k={k} L={L} spread={spread}")
    C = to_np(gpu_lib.dgemm_split(dev_cm(A), dev_cm(B), L))
    assert bits_equal(C, want)


@pytest.mark.parametrize("phi", [0.5, 4.0, 8.0])
def test_split_workload_law_bit_exact(gpu_lib, phi):
    m, n, k = 150, 170, 700
    A, B = dgemm_inputs(m, n, k, phi, SEED + int(phi * 10))
    want = o.dgemm_split2(A, B, 19)["C"]
    announce(f"dgemm_split workload law phi={phi}")
    assert bits_equal(to_np(gpu_lib.dgemm_split(dev_cm(A), dev_cm(B), 19)), want)


def test_split_equals_dgemm_when_one_term_is_exact(gpu_lib):
    """Integer inputs below 2^20 convert exactly in the first term (the
    second terms are 0), so the split route gives ozfp4_dgemm's C."""
    rng = np.random.default_rng(SEED + 2)
    A = rng.integers(-(1 << 20), 1 << 20, (120, 333)).astype(np.float64)
    B = rng.integers(-(1 << 20), 1 << 20, (333, 90)).astype(np.float64)
    announce("dgemm_split vs dgemm on exactly convertible inputs")
    Ad, Bd = dev_cm(A), dev_cm(B)
    assert bits_equal(to_np(gpu_lib.dgemm_split(Ad, Bd, 16)), to_np(gpu_lib.dgemm(Ad, Bd, 16)))


def test_split_edge_values(gpu_lib):
    rng = np.random.default_rng(SEED + 3)
    A = _wide(40, 50, 60, SEED + 4)
    B = _wide(50, 30, 60, SEED + 5)
    A[3, :] = 0.0                                   # zero row
    B[:, 4] = 0.0                                   # zero column
    A[5, :] = np.ldexp(A[5, :], -1070)              # a row of subnormals
    A[6, :] *= 2.0 ** 960                           # results beyond FP64: +-inf
    B[:, 7] *= 2.0 ** 100
    A[8, :] = 1.0
    B[:, 9] = 0.0
    B[0, 9], B[1, 9] = 2.0 ** 40, -(2.0 ** 40)      # exact cancellation
    A[10, :] = np.ldexp(A[10, :], -900)             # subnormal results
    B[:, 11] = np.ldexp(B[:, 11], -230)             # a subnormal result
    want = o.dgemm_split2(A, B, 19)["C"]
    announce("dgemm_split edge values")
    C = to_np(gpu_lib.dgemm_split(dev_cm(A), dev_cm(B), 19))
    assert bits_equal(C, want)
    assert np.isinf(C[6]).any() and (C[3] == 0).all() and C[8, 9] == 0.0
    assert ((C[10] != 0) & (np.abs(C[10]) < 2.0 ** -1022)).any()


def test_split_errors_and_empty(gpu_lib):
    import torch
    A = _wide(8, 9, 5, 1)
    B = _wide(9, 7, 5, 2)
    A[2, 3] = np.nan
    with pytest.raises(gpu_lib.OzFP4Error) as err:
        gpu_lib.dgemm_split(dev_cm(A), dev_cm(B), 19)
    assert err.value.code == gpu_lib.OZFP4_ENONFINITE
    Z = gpu_lib.dgemm_split(torch.zeros((5, 0), dtype=torch.float64, device="cuda"),
                            torch.zeros((0, 6), dtype=torch.float64, device="cuda"), 19)
    assert (to_np(Z) == 0).all() and Z.shape == (5, 6)


def test_split_largest_k(gpu_lib):
    """k = 131072: every product at its largest; the second terms
    adversarially at their bound (elements just below half an ulp of the
    first conversion)."""
    m, n, k = 3, 4, 131072
    rng = np.random.default_rng(SEED + 6)
    A = (1 + rng.random((m, k))) * np.where(rng.random((m, k)) < 0.5, -1.0, 1.0)
    B = (1 + rng.random((k, n))) * np.exp2(-rng.integers(0, 80, (k, n)))
    A[:, 0] = 2.0 ** 10                              # row maxima far above the rest
    announce(f"dgemm_split m={m} n={n} k={k}")
    want = o.dgemm_split2(A, B, 19)["C"]
    assert bits_equal(to_np(gpu_lib.dgemm_split(dev_cm(A), dev_cm(B), 19)), want)


def test_split_paper_law_phi32_correctly_rounded(gpu_lib):
    """The paper's input law at phi = 32 (Sec. VII-A: 128 x 128, K = 8192,
    19 moduli): every element of a line lies within 33 binades of its
    largest, inside c + d = 106 bits, so C = fl(AB) in all 16384 elements;
    the one-term route misses it."""
    A, B = paper_law_inputs(128, 128, 8192, 32, SEED + 7)
    announce("dgemm_split paper law phi=32, 128x128x8192")
    C = to_np(gpu_lib.dgemm_split(dev_cm(A), dev_cm(B), 19))
    ex, _ = o.exact_block(A, B, np.arange(128), np.arange(128))
    fl = np.array([[float(ex[i, j]) for j in range(128)] for i in range(128)])
    assert bits_equal(C, fl)
    assert bits_equal(C[:3, :3], o.dgemm_split2(A, B, 19, rows=np.arange(3), cols=np.arange(3))["C"])
    assert not bits_equal(to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), 19)), fl)


@pytest.mark.slow
def test_split_wide_workload_sampled(gpu_lib):
    """The wide-dynamic-range workload (m = n = 8192, k = 32768, phi = 4,
    19 moduli): sampled outputs bit for bit, and the normalized error of the
    sample within the final rounding (the one-term route reaches about
    2^-31 on this law)."""
    import torch
    M, K = 8192, 32768
    A, B = dgemm_inputs(M, M, K, 4.0, SEED + 8)
    rng = np.random.default_rng(4)
    rows = np.sort(rng.choice(M, 8, replace=False))
    cols = np.sort(rng.choice(M, 8, replace=False))
    announce("dgemm_split 8192 x 8192 x 32768 phi=4, sampled")
    C = gpu_lib.dgemm_split(dev_cm(A), dev_cm(B), 19)
    Cb = C[torch.as_tensor(rows, device="cuda")][:, torch.as_tensor(cols, device="cuda")].cpu().numpy()
    del C
    torch.cuda.empty_cache()
    want = o.dgemm_split2(A, B, 19, rows=rows, cols=cols)["C"]
    assert bits_equal(Cb, want)
    err = o.normalized_errors_block(Cb, A, B, rows, cols).max()
    announce(f"split phi=4 sample: {-math.log2(err) if err else float('inf'):.1f} bits")
    assert err <= 2.0 ** -52


@pytest.fixture
def heads_setting(gpu_lib):
    yield
    gpu_lib.ozfp4_set_one_limb_moduli(0)


@pytest.mark.parametrize("h,m,n,k,L,spread", [
    (1, 131, 67, 129, 19, 40), (5, 300, 300, 200, 21, 60), (5, 64, 80, 300, 6, 30),
    (4, 97, 31, 1000, 21, 10), (2, 33, 97, 64, 12, 200)])
def test_split_with_one_limb_heads_bit_exact(gpu_lib, heads_setting, h, m, n, k, L, spread):
    A, B = _wide(m, k, spread, SEED + 40 + m), _wide(k, n, spread, SEED + 41 + n)
    want = o.dgemm_split2(A, B, L, heads=h)["C"]
    announce(f"dgemm_split with {h} one-limb heads m={m} n={n} k={k} L={L}")
    assert gpu_lib.ozfp4_set_one_limb_moduli(h) == gpu_lib.OZFP4_OK
    C = to_np(gpu_lib.dgemm_split(dev_cm(A), dev_cm(B), L))
    assert bits_equal(C, want)


def test_split_four_heads_give_the_greedy_19_result(gpu_lib, heads_setting):
    """At k = 4096 the 21-moduli list with four heads has the 19 greedy
    moduli's capacities (53 / 53): the split route's C is the same bit for
    bit."""
    A, B = dgemm_inputs(256, 256, 4096, 4.0, SEED + 42)
    Ad, Bd = dev_cm(A), dev_cm(B)
    announce("dgemm_split, 19 greedy moduli against 4 heads and 21 moduli")
    gpu_lib.ozfp4_set_one_limb_moduli(0)
    g = to_np(gpu_lib.dgemm_split(Ad, Bd, 19))
    gpu_lib.ozfp4_set_one_limb_moduli(4)
    h = to_np(gpu_lib.dgemm_split(Ad, Bd, 21))
    assert bits_equal(g, h)
    assert bits_equal(g[:4, :4], o.dgemm_split2(A, B, 19, rows=np.arange(4), cols=np.arange(4))["C"])
