"""GPU parity over seeded random configurations: for each case a seeded
generator draws m, n, k (from 1 to 300, most of them ragged
against every tile), the number of moduli, the exponent spread phi of the
inputs, the capacity cap and the residue-GEMM route, and the library's C is
compared bit for bit with the oracle's. Scheme I, the FP32 emulation, INT8,
the two-term split route and the one-limb moduli list get their own draws. Each case prints its parameters before it runs,
so a failure names them."""

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, bits_equal, dev_cm, to_np
from oracle.sgemm_fp4 import capacity_bits_fp32, sgemm as oracle_sgemm
from oracle.one_limb_fp4 import dgemm_one_limb as oracle_one_limb
from oracle.split2_fp4 import dgemm_split2 as oracle_split2
from paper_2608_06812_amd.workloads import dgemm_inputs, int8_inputs

pytestmark = pytest.mark.gpu

SEED = 20261204
N_DGEMM, N_SGEMM, N_OZI, N_INT8, N_SPLIT, N_ONE = 40, 16, 16, 16, 16, 16


def _dim(rng):
    """Mostly ragged sizes up to 300 (more than one 256-line tile), sometimes
    1..3 or an exact multiple of 32."""
    u = rng.random()
    if u < 0.15:
        return int(rng.integers(1, 4))
    if u < 0.3:
        return int(32 * rng.integers(1, 11))
    return int(rng.integers(4, 301))


def _moduli_for(k, rng, cap_ok):
    """A random number of moduli that holds k (the smallest valid one if the
    draw is too small)."""
    L = int(rng.integers(2, 28))
    while not cap_ok(k, L):
        L += 1
    return L


def _dgemm_case(i):
    rng = np.random.default_rng([SEED, i])
    m, n, k = _dim(rng), _dim(rng), _dim(rng)
    cmax = 63 if rng.random() < 0.3 else 53
    kar = bool(rng.random() < 0.3)

    def cap_ok(k_, L_):
        try:
            o.capacity_bits(k_, o.select_moduli(L_), cmax=cmax)
            return True
        except ValueError:
            return False
    L = _moduli_for(k, rng, cap_ok)
    phi = float(rng.choice([0.0, 0.5, 2.0, 6.0]))
    return m, n, k, L, phi, cmax, kar, int(rng.integers(1 << 30))


@pytest.mark.parametrize("case", range(N_DGEMM))
def test_random_dgemm(gpu_lib, case):
    m, n, k, L, phi, cmax, kar, seed = _dgemm_case(case)
    A, B = dgemm_inputs(m, n, k, phi, seed)
    want = o.dgemm(A, B, L, cmax=cmax)["C"]
    announce(f"random dgemm case {case}: m={m} n={n} k={k} L={L} phi={phi} cmax={cmax} "
             f"karatsuba={kar} seed={seed}")
    try:
        gpu_lib.ozfp4_set_max_capacity(cmax)
        gpu_lib.ozfp4_set_karatsuba(kar)
        C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), L))
    finally:
        gpu_lib.ozfp4_set_karatsuba(False)
        gpu_lib.ozfp4_set_max_capacity(53)
    assert bits_equal(C, want)


@pytest.mark.parametrize("case", range(N_SGEMM))
def test_random_sgemm(gpu_lib, case):
    rng = np.random.default_rng([SEED + 1, case])
    m, n, k = _dim(rng), _dim(rng), _dim(rng)

    def cap_ok(k_, L_):
        try:
            capacity_bits_fp32(k_, o.select_moduli(L_))
            return True
        except ValueError:
            return False
    L = _moduli_for(k, rng, cap_ok)
    phi = float(rng.choice([0.0, 0.5, 2.0]))
    seed = int(rng.integers(1 << 30))
    A, B = dgemm_inputs(m, n, k, phi, seed)
    A, B = A.astype(np.float32), B.astype(np.float32)
    want = oracle_sgemm(A, B, L)["C"]
    announce(f"random sgemm case {case}: m={m} n={n} k={k} L={L} phi={phi} seed={seed}")
    import torch
    Ad = torch.from_numpy(np.ascontiguousarray(A.T)).cuda().t()
    Bd = torch.from_numpy(np.ascontiguousarray(B.T)).cuda().t()
    C = gpu_lib.sgemm(Ad, Bd, L).cpu().numpy()
    assert np.array_equal(C.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("case", range(N_OZI))
def test_random_ozi(gpu_lib, case):
    rng = np.random.default_rng([SEED + 2, case])
    m, n, k = _dim(rng), _dim(rng), _dim(rng)
    p = int(rng.integers(1, 16))
    phi = float(rng.choice([0.0, 0.5, 2.0]))
    seed = int(rng.integers(1 << 30))
    A, B = dgemm_inputs(m, n, k, phi, seed)
    want = o.dgemm_ozi(A, B, p)["C"]
    announce(f"random scheme-I case {case}: m={m} n={n} k={k} p={p} phi={phi} seed={seed}")
    C = to_np(gpu_lib.dgemm_ozi(dev_cm(A), dev_cm(B), p))
    assert bits_equal(C, want)


@pytest.mark.parametrize("case", range(N_INT8))
def test_random_igemm_s8(gpu_lib, case):
    import torch
    rng = np.random.default_rng([SEED + 3, case])
    m, n, k = _dim(rng), _dim(rng), _dim(rng) * int(rng.choice([1, 8]))
    seed = int(rng.integers(1 << 30))
    A, B = int8_inputs(m, n, k, seed)
    want = o.igemm_s8(A, B)
    announce(f"random igemm_s8 case {case}: m={m} n={n} k={k} seed={seed}")
    Ad = torch.from_numpy(np.ascontiguousarray(A.T)).cuda().t()
    Bd = torch.from_numpy(np.ascontiguousarray(B.T)).cuda().t()
    C = gpu_lib.igemm_s8(Ad, Bd).cpu().numpy()
    assert np.array_equal(C, want)


@pytest.mark.parametrize("case", range(N_SPLIT))
def test_random_split(gpu_lib, case):
    """The two-term split route (53-bit capacities), phi up to 12 so the
    second terms carry many bits."""
    rng = np.random.default_rng([SEED + 4, case])
    m, n, k = _dim(rng), _dim(rng), _dim(rng)

    def cap_ok(k_, L_):
        try:
            o.capacity_bits(k_, o.select_moduli(L_))
            return True
        except ValueError:
            return False
    L = _moduli_for(k, rng, cap_ok)
    phi = float(rng.choice([0.5, 4.0, 12.0]))
    seed = int(rng.integers(1 << 30))
    A, B = dgemm_inputs(m, n, k, phi, seed)
    want = oracle_split2(A, B, L)["C"]
    announce(f"random split case {case}: m={m} n={n} k={k} L={L} phi={phi} seed={seed}")
    C = to_np(gpu_lib.dgemm_split(dev_cm(A), dev_cm(B), L))
    assert bits_equal(C, want)


@pytest.mark.parametrize("case", range(N_ONE))
def test_random_one_limb(gpu_lib, case):
    """The one-limb moduli lists (1..5 heads) at caps 53 and 63."""
    rng = np.random.default_rng([SEED + 5, case])
    m, n, k = _dim(rng), _dim(rng), _dim(rng)
    cmax = 63 if rng.random() < 0.3 else 53
    h = int(rng.integers(1, 6))

    def cap_ok(k_, L_):
        try:
            o.capacity_bits(k_, o.select_moduli_one_limb(L_, heads=h), cmax=cmax)
            return True
        except ValueError:
            return False
    L = _moduli_for(k, rng, cap_ok)
    phi = float(rng.choice([0.0, 0.5, 2.0, 6.0]))
    seed = int(rng.integers(1 << 30))
    A, B = dgemm_inputs(m, n, k, phi, seed)
    want = oracle_one_limb(A, B, L, cmax=cmax, heads=h)["C"]
    announce(f"random one-limb case {case}: m={m} n={n} k={k} L={L} heads={h} phi={phi} "
             f"cmax={cmax} seed={seed}")
    try:
        gpu_lib.ozfp4_set_max_capacity(cmax)
        gpu_lib.ozfp4_set_one_limb_moduli(h)
        C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), L))
    finally:
        gpu_lib.ozfp4_set_one_limb_moduli(0)
        gpu_lib.ozfp4_set_max_capacity(53)
    assert bits_equal(C, want)
