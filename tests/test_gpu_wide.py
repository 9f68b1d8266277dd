"""GPU parity of the wide-range extension (ozfp4_set_max_capacity(63) with up
to 27 moduli): shifts, limb planes, residues and C against the oracle run
with the same cap, exactly; and the accuracy gain on the phi = 4 workload
(8192 x 8192 x 32768)."""

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, bits_equal, dev_cm, oracle_plane_codes, to_np, unpack_planes
from paper_2608_06812_amd.workloads import dgemm_inputs

pytestmark = pytest.mark.gpu

SEED = 20261006

# (m, n, k, L, phi)
SHAPES = [
    (131, 67, 129, 23, 4.0),
    (200, 130, 333, 21, 0.5),
    (64, 64, 1000, 27, 4.0),
    (1, 300, 77, 24, 4.0),
    (256, 256, 256, 22, 2.0),
]


@pytest.fixture
def wide(gpu_lib):
    assert gpu_lib.ozfp4_set_max_capacity(63) == 0
    try:
        yield gpu_lib
    finally:
        gpu_lib.ozfp4_set_max_capacity(53)


@pytest.mark.parametrize("m,n,k,L,phi", SHAPES)
def test_wide_scales_and_planes_exact(wide, m, n, k, L, phi):
    A, B = dgemm_inputs(m, n, k, phi, SEED)
    res = o.dgemm(A, B, L, cmax=63)
    assert max(res["cA"], res["cB"]) > 53
    announce(f"wide scales m={m} n={n} k={k} L={L}")
    s, t = wide.scales(dev_cm(A), dev_cm(B), L)
    assert np.array_equal(to_np(s), res["s"]) and np.array_equal(to_np(t), res["t"])
    announce(f"wide limb_planes m={m} n={n} k={k} L={L}")
    pa, pb = wide.limb_planes(dev_cm(A), dev_cm(B), L)
    ra, kp, _ = wide.ozfp4_plane_layout(m, k)
    rbp, _, _ = wide.ozfp4_plane_layout(n, k)
    assert np.array_equal(unpack_planes(to_np(pa), ra, kp),
                          oracle_plane_codes(res["Ai"], res["moduli"], ra, kp))
    assert np.array_equal(unpack_planes(to_np(pb), rbp, kp),
                          oracle_plane_codes(res["Bi"].T, res["moduli"], rbp, kp))


@pytest.mark.parametrize("m,n,k,L,phi", SHAPES)
def test_wide_residues_and_c_bit_exact(wide, m, n, k, L, phi):
    A, B = dgemm_inputs(m, n, k, phi, SEED + 1)
    res = o.dgemm(A, B, L, cmax=63)
    announce(f"wide residues m={m} n={n} k={k} L={L}")
    R = to_np(wide.residues(dev_cm(A), dev_cm(B), L))
    for l in range(L):
        assert np.array_equal(R[l].T.astype(np.int64), res["r"][l]), f"modulus {res['moduli'][l]}"
    announce(f"wide dgemm m={m} n={n} k={k} L={L}")
    C = to_np(wide.dgemm(dev_cm(A), dev_cm(B), L))
    assert bits_equal(C, res["C"])


def test_wide_edge_values(wide):
    """Zero lines, subnormal and huge values, exact cancellation, with
    63-bit capacities (23 moduli)."""
    rng = np.random.default_rng(SEED + 2)
    m, n, k = 70, 50, 90
    A = (rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-60, 60, size=(m, k)))
    B = (rng.random((k, n)) - 0.5) * np.exp2(rng.integers(-60, 60, size=(k, n)))
    A[0, :] = 0.0
    B[:, 1] = 0.0
    A[2, :] *= 1e-300
    A[4, :] = 1e300
    B[:, 5] = 1e300
    A[6, :5] = [5e-324, -5e-324, 1e-310, 2.5, 0.5]
    A[7, :] = 1.0
    B[:, 7] = 0.0
    B[0, 7], B[1, 7] = 1.0, -1.0
    want = o.dgemm(A, B, 23, cmax=63)
    assert (want["cA"], want["cB"]) == (63, 63)
    announce("wide dgemm edge values L=23")
    C = to_np(wide.dgemm(dev_cm(A), dev_cm(B), 23))
    assert bits_equal(C, want["C"])


@pytest.mark.slow
def test_wide_phi4_8192_sampled_and_more_accurate(gpu_lib):
    """The phi = 4 workload, m = n = 8192, k = 32768: with 23 moduli and
    63-bit capacities, sampled outputs equal the oracle's bit for bit, and
    the normalized error on a sample drops well below the 19-moduli, 53-bit
    result's."""
    import torch
    m = n = 8192
    k = 32768
    A, B = dgemm_inputs(m, n, k, 4.0, SEED + 3)
    rows = np.array([0, 1, 777, 4095, 8191])
    cols = np.array([0, 5, 2048, 6000, 8191])
    Ad, Bd = dev_cm(A), dev_cm(B)
    errs = {}
    for L, cmax in ((19, 53), (23, 63)):
        gpu_lib.ozfp4_set_max_capacity(cmax)
        try:
            announce(f"dgemm phi=4 8192x8192x32768 L={L} cmax={cmax}")
            Cd = gpu_lib.dgemm(Ad, Bd, L)
            C = to_np(Cd[torch.as_tensor(rows, device="cuda")][:, torch.as_tensor(cols, device="cuda")])
            del Cd
        finally:
            gpu_lib.ozfp4_set_max_capacity(53)
        want = o.dgemm(A, B, L, rows=rows, cols=cols, cmax=cmax)
        assert bits_equal(C, want["C"])
        errs[cmax] = max(o.normalized_error(C[i, j], A, B, int(rows[i]), int(cols[j]))
                         for i in range(len(rows)) for j in range(len(cols)))
    announce(f"normalized error: 53-bit {errs[53]:.3e}, 63-bit {errs[63]:.3e}")
    assert errs[63] * 2 ** 6 <= errs[53]


@pytest.mark.slow
def test_wide_at_the_largest_k(wide):
    """k = 131072 (OZFP4_MAX_K) with all 27 moduli and 63-bit capacities
    (four CRT chunks, the exact path for every element): residues and C bit
    for bit against the oracle, on wide exponents and on lines of equal
    largest values."""
    m, n, k, L = 24, 16, wide.OZFP4_MAX_K, 27
    A, B = dgemm_inputs(m, n, k, 4.0, SEED + 5)
    A[0, :] = 1.0 - 2.0 ** -53
    B[:, 0] = -(1.0 - 2.0 ** -53)
    res = o.dgemm(A, B, L, cmax=63)
    assert (res["cA"], res["cB"]) == (63, 63)
    announce(f"wide residues and dgemm k={k} L={L}")
    R = to_np(wide.residues(dev_cm(A), dev_cm(B), L))
    for l in range(L):
        assert np.array_equal(R[l].T.astype(np.int64), res["r"][l]), f"modulus {res['moduli'][l]}"
    C = to_np(wide.dgemm(dev_cm(A), dev_cm(B), L))
    assert bits_equal(C, res["C"])
