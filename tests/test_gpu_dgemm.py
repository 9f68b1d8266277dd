"""GPU parity of the Ozaki-II-on-FP4 DGEMM path against the CPU oracle.

Every comparison is exact: shifts, packed limb planes (byte for byte),
residue matrices and C (bit for bit). Inputs are seeded synthetic matrices
from paper_2608_06812_amd.workloads; the oracle never sees GPU output as
input."""

import math

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, bits_equal, dev_cm, oracle_plane_codes, to_np, unpack_planes
from paper_2608_06812_amd.workloads import dgemm_inputs, paper_law_inputs

pytestmark = pytest.mark.gpu

SEED = 20260806

# (m, n, k, L): several tiles, ragged tails, degenerate sizes
SHAPES = [
    (256, 256, 256, 14),       # the small configuration, full output
    (131, 67, 129, 19),        # ragged in every dimension
    (1, 1, 1, 19),
    (1, 300, 77, 16),
    (300, 1, 200, 12),
    (200, 130, 333, 20),
    (64, 64, 1000, 17),
]


def _inputs(m, n, k, phi=0.5, seed=SEED):
    return dgemm_inputs(m, n, k, phi, seed)


@pytest.mark.parametrize("m,n,k,L", SHAPES)
def test_scales_exact(gpu_lib, m, n, k, L):
    A, B = _inputs(m, n, k)
    cA, cB = o.capacity_bits(k, o.select_moduli(L))
    announce(f"scales m={m} n={n} k={k} L={L}")
    s, t = gpu_lib.scales(dev_cm(A), dev_cm(B), L)
    assert np.array_equal(to_np(s), o.shift_exponents(A, axis=1, c=cA))
    assert np.array_equal(to_np(t), o.shift_exponents(B, axis=0, c=cB))


@pytest.mark.parametrize("m,n,k,L", [(131, 67, 129, 19), (64, 40, 300, 14), (33, 97, 64, 20)])
def test_limb_planes_byte_exact(gpu_lib, m, n, k, L):
    A, B = _inputs(m, n, k, seed=SEED + 7)
    res = o.dgemm(A[:, :], B, L, rows=np.arange(m), cols=np.arange(n))
    moduli = res["moduli"]
    announce(f"limb_planes m={m} n={n} k={k} L={L}")
    pa, pb = gpu_lib.limb_planes(dev_cm(A), dev_cm(B), L)
    ra, kp, _ = gpu_lib.ozfp4_plane_layout(m, k)
    rbp, _, _ = gpu_lib.ozfp4_plane_layout(n, k)
    got_a = unpack_planes(to_np(pa), ra, kp)
    got_b = unpack_planes(to_np(pb), rbp, kp)
    want_a = oracle_plane_codes(res["Ai"], moduli, ra, kp)
    want_b = oracle_plane_codes(res["Bi"].T, moduli, rbp, kp)
    assert np.array_equal(got_a, want_a)
    assert np.array_equal(got_b, want_b)


@pytest.mark.parametrize("m,n,k,L", SHAPES)
def test_residues_bit_exact(gpu_lib, m, n, k, L):
    A, B = _inputs(m, n, k, seed=SEED + 1)
    res = o.dgemm(A, B, L)
    announce(f"residues m={m} n={n} k={k} L={L}")
    R = to_np(gpu_lib.residues(dev_cm(A), dev_cm(B), L))
    for l in range(L):
        assert np.array_equal(R[l].T.astype(np.int64), res["r"][l]), f"modulus {res['moduli'][l]}"


@pytest.mark.parametrize("m,n,k,L", SHAPES)
def test_dgemm_bit_exact(gpu_lib, m, n, k, L):
    A, B = _inputs(m, n, k, seed=SEED + 2)
    want = o.dgemm(A, B, L)["C"]
    announce(f"dgemm m={m} n={n} k={k} L={L}")
    C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), L))
    assert bits_equal(C, want)


def test_dgemm_edge_values(gpu_lib):
    """Zero rows and columns, subnormal inputs and outputs, overflow to inf,
    exact cancellation, ties in the conversion."""
    rng = np.random.default_rng(SEED + 3)
    m, n, k = 70, 50, 90
    A = (rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-20, 20, size=(m, k)))
    B = (rng.random((k, n)) - 0.5) * np.exp2(rng.integers(-20, 20, size=(k, n)))
    A[0, :] = 0.0
    B[:, 1] = 0.0
    A[2, :] *= 1e-300                      # subnormal products
    B[:, 3] *= 1e-20
    A[4, :] = 1e300                        # overflow to +-inf with large columns
    B[:, 5] = 1e300
    A[6, :5] = [5e-324, -5e-324, 1e-310, 2.5, 0.5]
    A[7, :] = 1.0
    B[:, 7] = 0.0
    B[0, 7], B[1, 7] = 1.0, -1.0          # exact cancellation in row 7, column 7
    for L in (14, 19):
        want = o.dgemm(A, B, L)["C"]
        announce(f"dgemm edge values L={L}")
        C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), L))
        assert bits_equal(C, want)
        assert np.isinf(C[4, 5]) and np.any(C[2, :] != 0) and np.all(C[0, :] == 0)


def test_dgemm_k_zero_and_empty(gpu_lib):
    import torch
    A = dev_cm(np.zeros((5, 0)))
    B = dev_cm(np.zeros((0, 4)))
    announce("dgemm k=0")
    C = gpu_lib.dgemm(A, B, 19)
    assert C.shape == (5, 4) and bool(torch.all(C == 0))
    announce("dgemm m=0")
    C0 = gpu_lib.dgemm(dev_cm(np.zeros((0, 3))), dev_cm(np.ones((3, 2))), 19)
    assert C0.shape == (0, 2)


def test_dgemm_nonfinite_is_reported(gpu_lib):
    A, B = _inputs(40, 30, 20)
    for bad in (np.nan, np.inf, -np.inf):
        A2 = A.copy()
        A2[3, 4] = bad
        announce(f"dgemm non-finite A {bad}")
        with pytest.raises(gpu_lib.OzFP4Error) as ei:
            gpu_lib.dgemm(dev_cm(A2), dev_cm(B), 19)
        assert ei.value.code == gpu_lib.OZFP4_ENONFINITE
        B2 = B.copy()
        B2[5, 6] = bad
        announce(f"dgemm non-finite B {bad}")
        with pytest.raises(gpu_lib.OzFP4Error):
            gpu_lib.dgemm(dev_cm(A), dev_cm(B2), 19)
    # a clean call afterwards still works (the flag is cleared per call)
    announce("dgemm after non-finite")
    C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), 19))
    assert bits_equal(C, o.dgemm(A, B, 19)["C"])


def test_dgemm_leading_dimensions(gpu_lib):
    """Sub-matrix views: lda, ldb, ldc larger than the row counts."""
    import torch
    m, n, k = 90, 70, 150
    A, B = _inputs(m, n, k, seed=SEED + 4)
    Abig = np.zeros((m + 13, k))
    Abig[:m] = A
    Bbig = np.zeros((k + 5, n))
    Bbig[:k] = B
    Ad = dev_cm(Abig)[:m]
    Bd = dev_cm(Bbig)[:k]
    out = torch.full((m + 3, n), 7.0, dtype=torch.float64, device="cuda").t().contiguous().t()
    announce("dgemm leading dimensions")
    gpu_lib.dgemm(Ad, Bd, 19, out=out[:m])
    got = to_np(out)
    assert bits_equal(got[:m], o.dgemm(A, B, 19)["C"])
    assert np.all(got[m:] == 7.0)


def test_dgemm_phi0_is_correctly_rounded(gpu_lib):
    """Paper law at phi = 0 with L = 19: the conversion is exact, so C must
    equal the correctly rounded fl(AB) (Sec. VII-A)."""
    A, B = paper_law_inputs(48, 40, 512, phi=0, seed=SEED + 5)
    announce("dgemm phi=0 paper law")
    C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), 19))
    for i in range(0, 48, 5):
        for j in range(0, 40, 3):
            assert C[i, j] == float(o.exact_product_entry(A, B, i, j))


def test_residues_adversarial_exactness_at_max_k(gpu_lib):
    """FP32 accumulators at the exactness limit (k = 131072): every limb of
    modulus 169 is +8 (residue 112 splits as (8, 8)), so the cross-term
    accumulator reaches 2^22 in units of the stored values, and the last k
    adds products of limbs 1 x 1 (a quarter) that an inexact accumulation
    would drop. Residues of every modulus must still equal the oracle's."""
    k = 131072
    m = n = 64
    assert o.two_limb_split(112, 169) == (8, 8)
    # integers below 2^52 with the line maxima in [2^52, 2^53) (A, c = 53)
    # and [2^51, 2^52) (B, c = 52) convert exactly (shift 0)
    A = np.full((m, k), 112.0 + 169.0 * 1000)
    B = np.full((k, n), 112.0 + 169.0 * 7)
    A[:, 0] = 2.0 ** 52 + 169 * np.arange(m)      # row maxima
    B[0, :] = 2.0 ** 51 + 169 * np.arange(n)      # column maxima
    A[:, -3:] = 1.0
    B[-3:, :] = 1.0
    A[:5, 1:9] = -112.0                             # some rows flip sign early
    assert o.capacity_bits(k, o.select_moduli(19)) == (53, 52)
    res = o.dgemm(A, B, 19)
    assert np.array_equal(res["Ai"], A.astype(np.int64))
    announce("residues adversarial k=131072")
    R = to_np(gpu_lib.residues(dev_cm(A), dev_cm(B), 19))
    for l in range(19):
        assert np.array_equal(R[l].T.astype(np.int64), res["r"][l]), f"modulus {res['moduli'][l]}"
    announce("dgemm adversarial k=131072")
    C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), 19))
    assert bits_equal(C, res["C"])


def _sampled_check(gpu_lib, A, B, L, rows, cols, accuracy_sample=0):
    import torch
    announce(f"dgemm sampled m={A.shape[0]} n={B.shape[1]} k={A.shape[1]} L={L}")
    Ad, Bd = dev_cm(A), dev_cm(B)
    Cd = gpu_lib.dgemm(Ad, Bd, L)
    assert bool(torch.isfinite(Cd).all())
    C = to_np(Cd[torch.as_tensor(rows, device="cuda")][:, torch.as_tensor(cols, device="cuda")])
    del Ad, Bd, Cd
    want = o.dgemm(A, B, L, rows=rows, cols=cols)
    assert bits_equal(C, want["C"])
    worst = 0.0
    for i in range(min(accuracy_sample, len(rows))):
        for j in range(min(accuracy_sample, len(cols))):
            worst = max(worst, o.normalized_error(C[i, j], A, B, int(rows[i]), int(cols[j])))
    return worst


@pytest.mark.slow
def test_dgemm_4096_sampled_and_accurate(gpu_lib):
    """Config m = n = k = 4096 with L = 18 (the smallest L that meets the
    FP64 accuracy target there): sampled outputs bit-exact, normalized error
    below 2^-50 on a sample."""
    A, B = dgemm_inputs(4096, 4096, 4096, 0.5, SEED + 10)
    rng = np.random.default_rng(1)
    rows = np.sort(rng.choice(4096, 24, replace=False))
    cols = np.sort(rng.choice(4096, 24, replace=False))
    worst = _sampled_check(gpu_lib, A, B, 18, rows, cols, accuracy_sample=4)
    assert worst <= 2.0 ** -50


@pytest.mark.slow
def test_dgemm_16384_sampled(gpu_lib):
    """The benchmark configuration (m = n = k = 16384, L = 18), sampled."""
    A, B = dgemm_inputs(16384, 16384, 16384, 0.5, SEED + 20)
    rng = np.random.default_rng(2)
    rows = np.concatenate([[0, 16383], np.sort(rng.choice(16384, 10, replace=False))])
    cols = np.concatenate([[0, 16383], np.sort(rng.choice(16384, 10, replace=False))])
    _sampled_check(gpu_lib, A, B, 18, rows, cols)


@pytest.mark.slow
def test_dgemm_wide_range_sampled(gpu_lib):
    """m = n = 8192, k = 32768, phi = 4 (large exponent spread), L = 19:
    sampled outputs bit-exact, and within the a-priori bound of the
    shared-exponent quantization."""
    A, B = dgemm_inputs(8192, 8192, 32768, 4.0, SEED + 30)
    rng = np.random.default_rng(3)
    rows = np.sort(rng.choice(8192, 8, replace=False))
    cols = np.sort(rng.choice(8192, 8, replace=False))
    _sampled_check(gpu_lib, A, B, 19, rows, cols)
    want = o.dgemm(A, B, 19, rows=rows, cols=cols)
    bound = o.quantization_error_bound(A, B, want["s"], want["t"], want["x"], rows, cols)
    exact, _ = o.exact_block(A, B, rows, cols)
    from fractions import Fraction
    for i in range(len(rows)):
        for j in range(len(cols)):
            err = abs(Fraction(float(want["C"][i, j])) - exact[i, j])
            assert err <= Fraction(float(bound[i, j])), (i, j)


@pytest.mark.slow
@pytest.mark.parametrize("phi,key", [(0, "accuracy_bits_phi0"), (32, "accuracy_bits_phi32")])
def test_paper_accuracy_experiment(gpu_lib, paper, phi, key):
    """Sec. VII-A: the paper's input law at K = 8192, a whole 128 x 128
    output, 19 moduli; the maximum normalized error over all 16384 outputs
    (exact reference) is within 0.75 bit of the printed value."""
    import math
    A, B = paper_law_inputs(128, 128, 8192, phi, SEED + 60 + phi)
    announce(f"dgemm paper accuracy phi={phi}")
    C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), 19))
    assert bits_equal(C[:4, :4], o.dgemm(A, B, 19, rows=np.arange(4), cols=np.arange(4))["C"])
    err = o.normalized_errors_block(C, A, B, np.arange(128), np.arange(128)).max()
    bits = -math.log2(err)
    announce(f"phi={phi}: {bits:.2f} bits (paper {paper[key]})")
    assert abs(bits - paper[key]) <= 0.75


@pytest.mark.slow
def test_residues_16384_full_for_two_moduli(gpu_lib):
    """The benchmark workload (m = n = k = 16384, L = 18): every one of the
    2^28 residues of modulus 169 (whose tile skips the a1 b1 products, as
    13^2 = 0 mod 169) and of modulus 115 (the modulus with the paper's worked
    split, -58 = 13 (-4) - 6) equals the definition (A~ B~) mod m, formed
    from the oracle's converted integers as ((A~ mod m)(B~ mod m)) mod m by
    one FP64 product, exact because every sum is below 168^2 k < 2^53."""
    import torch
    N, L = 16384, 18
    A, B = dgemm_inputs(N, N, N, 0.5, SEED + 11)
    moduli = o.select_moduli(L)
    assert moduli[:2] == [169, 115]
    cA, cB = o.capacity_bits(N, moduli)
    Ai = o.to_integers(A, o.shift_exponents(A, axis=1, c=cA), axis=1)
    Bi = o.to_integers(B, o.shift_exponents(B, axis=0, c=cB), axis=0)
    announce("residues 16384^3 L=18, all of moduli 169 and 115")
    Ad, Bd = dev_cm(A), dev_cm(B)
    del A, B
    R = gpu_lib.residues(Ad, Bd, L)
    got = [R[i].cpu().numpy().T for i in (0, 1)]   # (m, n) each
    del R, Ad, Bd
    torch.cuda.empty_cache()
    assert 168.0 ** 2 * N < 2.0 ** 53
    for i, m in ((0, 169), (1, 115)):
        ra = o.residues(Ai, m).astype(np.float64)
        rb = o.residues(Bi, m).astype(np.float64)
        want = np.mod(np.rint(ra @ rb).astype(np.int64), m)
        del ra, rb
        assert got[i].shape == want.shape
        assert np.array_equal(got[i].astype(np.int64), want), f"modulus {m}"
