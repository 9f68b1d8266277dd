"""GPU parity of the Karatsuba mode (ozfp4_set_karatsuba(1), Sec. V-A): the
Karatsuba moduli run three limb products from the sum-limb split and a third
operand plane. Limb planes are compared byte for byte with the oracle's
sum-limb planes; residues and C bit for bit with the oracle (which are the
same as in the default mode)."""

import math

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, bits_equal, dev_cm, oracle_plane_codes, to_np, unpack_planes
from paper_2608_06812_amd.workloads import dgemm_inputs

pytestmark = pytest.mark.gpu

SEED = 20260906

SHAPES = [
    (256, 256, 256, 14),
    (131, 67, 129, 19),
    (1, 1, 1, 19),
    (200, 130, 333, 20),
    (64, 64, 1000, 17),
    (300, 1, 200, 12),
]


@pytest.fixture
def kar(gpu_lib):
    gpu_lib.ozfp4_set_karatsuba(True)
    try:
        yield gpu_lib
    finally:
        gpu_lib.ozfp4_set_karatsuba(False)


@pytest.mark.parametrize("m,n,k,L", [(131, 67, 129, 19), (33, 97, 64, 20), (64, 40, 300, 14)])
def test_karatsuba_limb_planes_byte_exact(kar, m, n, k, L):
    A, B = dgemm_inputs(m, n, k, 0.5, SEED)
    res = o.dgemm(A, B, L)
    moduli = res["moduli"]
    announce(f"karatsuba limb_planes m={m} n={n} k={k} L={L}")
    pa, pb = kar.limb_planes(dev_cm(A), dev_cm(B), L)
    assert pa.shape[0] == 2 * L + len(o.karatsuba_moduli(moduli))
    ra, kp, _ = kar.ozfp4_plane_layout(m, k)
    rbp, _, _ = kar.ozfp4_plane_layout(n, k)
    assert np.array_equal(unpack_planes(to_np(pa), ra, kp),
                          oracle_plane_codes(res["Ai"], moduli, ra, kp, karatsuba=True))
    assert np.array_equal(unpack_planes(to_np(pb), rbp, kp),
                          oracle_plane_codes(res["Bi"].T, moduli, rbp, kp, karatsuba=True))


@pytest.mark.parametrize("m,n,k,L", SHAPES)
def test_karatsuba_residues_bit_exact(kar, m, n, k, L):
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 1)
    res = o.dgemm(A, B, L, karatsuba=True)
    announce(f"karatsuba residues m={m} n={n} k={k} L={L}")
    R = to_np(kar.residues(dev_cm(A), dev_cm(B), L))
    for l in range(L):
        assert np.array_equal(R[l].T.astype(np.int64), res["r"][l]), f"modulus {res['moduli'][l]}"


@pytest.mark.parametrize("m,n,k,L", SHAPES)
def test_karatsuba_dgemm_bit_exact(kar, m, n, k, L):
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 2)
    want = o.dgemm(A, B, L)["C"]
    announce(f"karatsuba dgemm m={m} n={n} k={k} L={L}")
    C = to_np(kar.dgemm(dev_cm(A), dev_cm(B), L))
    assert bits_equal(C, want)


def test_karatsuba_adversarial_k_max(kar):
    """k = 131072 with every value = 8 modulo the product of the Karatsuba
    moduli among 19: each of them splits 8 as (8, 0), sum 8, so P0 and Ps
    reach 2^21 in units of the stored values, and the last k add quarter
    products that an inexact FP32 accumulation would drop."""
    k = 131072
    m = n = 64
    moduli = o.select_moduli(19)
    kmods = o.karatsuba_moduli(moduli)
    for mod in kmods:
        assert o.sum_limb_split(8, mod) == (8, 0)
    Pk = math.prod(kmods)
    assert 8 + 5 * Pk < 2 ** 51
    A = np.full((m, k), float(8 + 3 * Pk))
    B = np.full((k, n), float(8 + 5 * Pk))
    A[:, 0] = 2.0 ** 52 + Pk * np.arange(m) + 8      # row maxima, c = 53
    B[0, :] = 2.0 ** 51 + Pk * np.arange(n) + 8      # column maxima, c = 52
    A[:, -3:] = 1.0
    B[-3:, :] = 1.0
    A[:5, 1:9] = -8.0
    assert o.capacity_bits(k, moduli) == (53, 52)
    res = o.dgemm(A, B, 19)
    assert np.array_equal(res["Ai"], A.astype(np.int64))
    announce("karatsuba residues adversarial k=131072")
    R = to_np(kar.residues(dev_cm(A), dev_cm(B), 19))
    for l in range(19):
        assert np.array_equal(R[l].T.astype(np.int64), res["r"][l]), f"modulus {res['moduli'][l]}"
    announce("karatsuba dgemm adversarial k=131072")
    C = to_np(kar.dgemm(dev_cm(A), dev_cm(B), 19))
    assert bits_equal(C, res["C"])


def test_modes_agree_on_c(gpu_lib):
    """The same call in both modes gives bitwise the same C (ragged shape)."""
    A, B = dgemm_inputs(300, 170, 700, 0.5, SEED + 3)
    Ad, Bd = dev_cm(A), dev_cm(B)
    announce("dgemm default mode 300x170x700 L=18")
    C0 = to_np(gpu_lib.dgemm(Ad, Bd, 18))
    gpu_lib.ozfp4_set_karatsuba(True)
    try:
        announce("dgemm karatsuba mode 300x170x700 L=18")
        C1 = to_np(gpu_lib.dgemm(Ad, Bd, 18))
    finally:
        gpu_lib.ozfp4_set_karatsuba(False)
    assert bits_equal(C0, C1)
