"""GPU parity of the one-limb moduli lists (ozfp4_set_one_limb_moduli(h):
the first h of 11, 9, 8, 7, 5 with one limb each, then the greedy rule
seeded with them; mostly h = 1, 11 then the greedy moduli) against the oracle
(oracle/one_limb_fp4.py): the scales, the limb planes byte for byte, every
residue plane (11's from the single-product GEMM, the others from the
default GEMM), and C bit for bit, on ragged shapes, shapes whose tile grid
takes the XCD-share mapping of both GEMMs, edge values, the largest k, the
wide capacity cap, the allocation-free entry point, the FP32 emulation over
the list, and sampled outputs of m = n = k = 16384 with 18 moduli, whose
normalized error must stay within 2^-50. With 2..5 heads: C bit for bit
(including lists of heads only), every residue plane, and C equal to the
greedy 18 / 19 moduli's C where the capacities agree."""

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, bits_equal, dev_cm, to_np, unpack_planes
from paper_2608_06812_amd.workloads import dgemm_inputs

pytestmark = pytest.mark.gpu

SEED = 20261401


@pytest.fixture(autouse=True)
def one_limb(gpu_lib):
    assert gpu_lib.ozfp4_set_one_limb_moduli(1) == gpu_lib.OZFP4_OK
    yield
    gpu_lib.ozfp4_set_one_limb_moduli(0)
    gpu_lib.ozfp4_set_max_capacity(53)


SHAPES = [
    (1, 1, 1, 18),
    (131, 67, 129, 18),       # ragged in every dimension
    (300, 300, 200, 18),      # 2 x 4 tiles of the default GEMM: the XCD-share mapping
    (1000, 200, 300, 19),     # 4 x 2 tiles
    (97, 31, 1000, 14),
    (513, 257, 130, 20),
    (256, 256, 100, 2),       # 11 and 169 only: capacities 2 / 1
    (64, 700, 64, 27),
]


@pytest.mark.parametrize("m,n,k,L", SHAPES)
def test_one_limb_dgemm_bit_exact(gpu_lib, m, n, k, L):
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + m + n)
    want = o.dgemm_one_limb(A, B, L)["C"]
    announce(f"one-limb dgemm m={m} n={n} k={k} L={L}")
    C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), L))
    assert bits_equal(C, want)


@pytest.mark.parametrize("m,n,k,L", [(131, 67, 129, 18), (300, 300, 200, 19), (64, 40, 1000, 3)])
def test_one_limb_residues_bit_exact(gpu_lib, m, n, k, L):
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 1)
    res = o.dgemm_one_limb(A, B, L)
    announce(f"one-limb residues m={m} n={n} k={k} L={L}")
    R = to_np(gpu_lib.residues(dev_cm(A), dev_cm(B), L))
    for l in range(L):
        assert np.array_equal(R[l].T.astype(np.int64), res["r"][l]), f"modulus {res['moduli'][l]}"


def test_one_limb_scales_and_planes_byte_exact(gpu_lib):
    m, n, k, L = 131, 67, 300, 18
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 2)
    res = o.dgemm_one_limb(A, B, L)
    announce(f"one-limb scales and planes m={m} n={n} k={k} L={L}")
    s, t = gpu_lib.scales(dev_cm(A), dev_cm(B), L)
    assert np.array_equal(to_np(s), res["s"]) and np.array_equal(to_np(t), res["t"])
    pa, pb = gpu_lib.limb_planes(dev_cm(A), dev_cm(B), L)
    ra, kp, _ = gpu_lib.ozfp4_plane_layout(m, k)
    rb, _, _ = gpu_lib.ozfp4_plane_layout(n, k)
    got = [unpack_planes(to_np(pa), ra, kp), unpack_planes(to_np(pb), rb, kp)]
    code = np.vectorize(o.e2m1_code, otypes=[np.uint8])
    for X, G, rows in ((res["Ai"], got[0], ra), (res["Bi"].T, got[1], rb)):
        lines = X.shape[0]
        want = np.zeros((2 * L, rows, kp), dtype=np.uint8)
        want[0, :lines, :k] = code(o.one_limb_plane(X, 11))
        for l, q in enumerate(res["moduli"][1:], start=1):
            c0, c1 = o.limb_planes(X, q)
            want[2 * l, :lines, :k] = code(c0)
            want[2 * l + 1, :lines, :k] = code(c1)
        assert np.array_equal(G, want)


def test_one_limb_edge_values(gpu_lib):
    rng = np.random.default_rng(SEED + 3)
    m, n, k = 70, 50, 90
    A = (rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-20, 20, size=(m, k)))
    B = (rng.random((k, n)) - 0.5) * np.exp2(rng.integers(-20, 20, size=(k, n)))
    A[0, :] = 0.0
    B[:, 1] = 0.0
    A[2, :] *= 1e-300
    A[4, :] = 1e300
    B[:, 5] = 1e300
    A[6, :5] = [5e-324, -5e-324, 1e-310, 2.5, 0.5]
    A[7, :] = 1.0
    B[:, 7] = 0.0
    B[0, 7], B[1, 7] = 1.0, -1.0
    want = o.dgemm_one_limb(A, B, 18)["C"]
    announce("one-limb dgemm edge values")
    C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), 18))
    assert bits_equal(C, want)
    assert np.isinf(C[4, 5]) and np.all(C[0, :] == 0) and C[7, 7] == 0.0


def test_one_limb_largest_k(gpu_lib):
    """k = 131072 with 19 moduli (capacities 51 / 51): lines all equal to
    1.046875 = 67 / 64 convert to 67 2^44 = 5 (mod 11), so every one-limb
    code of row 0 of A and column 0 of B is -6 and the single-product
    accumulator reaches its bound 9 k; C(0, 0) = (67 / 64)^2 k exactly."""
    m, n, k = 3, 4, 131072
    rng = np.random.default_rng(SEED + 4)
    A = (1 + rng.random((m, k))) * np.where(rng.random((m, k)) < 0.5, -1.0, 1.0)
    B = 1 + rng.random((k, n))
    x = 67 / 64
    A[0, :] = x
    A[1, :] = -x
    B[:, 0] = x
    B[1::2, 1] = -x
    B[0::2, 1] = x
    res = o.dgemm_one_limb(A, B, 19, check_definition=True)
    assert (res["cA"], res["cB"]) == (51, 51)
    assert np.all(o.one_limb_plane(res["Ai"][:1], 11) == -6)
    assert np.all(o.one_limb_plane(res["Bi"][:, :1], 11) == -6)
    announce(f"one-limb dgemm m={m} n={n} k={k}")
    C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), 19))
    assert bits_equal(C, res["C"])
    assert C[0, 0] == x * x * k and C[1, 0] == -x * x * k and C[0, 1] == 0.0


def test_one_limb_wide_cap(gpu_lib):
    assert gpu_lib.ozfp4_set_max_capacity(63) == gpu_lib.OZFP4_OK
    A, B = dgemm_inputs(200, 130, 333, 4.0, SEED + 5)
    want = o.dgemm_one_limb(A, B, 24, cmax=63)["C"]
    announce("one-limb dgemm cap 63, L=24")
    assert bits_equal(to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), 24)), want)


def test_one_limb_noalloc_matches(gpu_lib):
    import torch
    assert gpu_lib.ozfp4_init() == gpu_lib.OZFP4_OK
    A, B = dgemm_inputs(300, 260, 500, 0.5, SEED + 6)
    announce("one-limb dgemm_noalloc vs dgemm")
    Ad, Bd = dev_cm(A), dev_cm(B)
    ref = to_np(gpu_lib.dgemm(Ad, Bd, 18))
    out = torch.empty_strided((300, 260), (1, 300), dtype=torch.float64, device="cuda")
    gpu_lib.dgemm_noalloc(Ad, Bd, out, 18)
    assert bits_equal(to_np(out), ref)
    assert bits_equal(ref, o.dgemm_one_limb(A, B, 18)["C"])


@pytest.mark.parametrize("m,n,k,L", [(131, 67, 129, 10), (300, 300, 200, 10), (64, 700, 64, 19),
                                     (1, 1, 1, 10)])
def test_one_limb_sgemm_bit_exact(gpu_lib, m, n, k, L):
    A, B = dgemm_inputs(m, n, k, 2.0, SEED + 10 + m)
    A, B = A.astype(np.float32), B.astype(np.float32)
    want = o.sgemm_one_limb(A, B, L)["C"]
    announce(f"one-limb sgemm m={m} n={n} k={k} L={L}")
    C = to_np(gpu_lib.sgemm(dev_cm(A), dev_cm(B), L))
    assert C.dtype == np.float32 and np.array_equal(C.view(np.uint32), want.view(np.uint32))


def test_one_limb_too_few_moduli_refused(gpu_lib):
    """P = 11 * 169 cannot hold k = 384 (b < 2): the oracle refuses and the
    library reports OZFP4_EMODULI before any GPU work."""
    A, B = dgemm_inputs(8, 8, 384, 0.5, SEED + 9)
    with pytest.raises(ValueError):
        o.dgemm_one_limb(A, B, 2)
    with pytest.raises(gpu_lib.OzFP4Error) as ei:
        gpu_lib.dgemm(dev_cm(A), dev_cm(B), 2)
    assert ei.value.code == gpu_lib.OZFP4_EMODULI


def test_one_limb_off_restores_the_greedy_list(gpu_lib):
    A, B = dgemm_inputs(96, 80, 200, 0.5, SEED + 7)
    gpu_lib.ozfp4_set_one_limb_moduli(0)
    announce("dgemm after the one-limb setting is cleared")
    assert bits_equal(to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), 14)), o.dgemm(A, B, 14)["C"])


def test_one_limb_residues_4096_every_modulus_full(gpu_lib):
    """m = n = k = 4096 with 18 moduli of the one-limb list: all 2^24
    residues of every modulus (11's from k_gemm_one_limb over 16 x 16 tiles,
    the others from k_gemm_res over 16 x 32 tiles per modulus) against
    ((A~ mod m)(B~ mod m)) mod m from the oracle's converted integers, one
    exact CPU FP64 product per modulus."""
    N, L = 4096, 18
    A, B = dgemm_inputs(N, N, N, 0.5, SEED + 11)
    moduli = o.select_moduli_one_limb(L)
    cA, cB = o.capacity_bits(N, moduli)
    Ai = o.to_integers(A, o.shift_exponents(A, axis=1, c=cA), axis=1)
    Bi = o.to_integers(B, o.shift_exponents(B, axis=0, c=cB), axis=0)
    announce("one-limb residues 4096^3 L=18, every modulus in full")
    R = to_np(gpu_lib.residues(dev_cm(A), dev_cm(B), L))
    assert 168.0 ** 2 * N < 2.0 ** 53
    for l, m in enumerate(moduli):
        ra = o.residues(Ai, m).astype(np.float64)
        rb = o.residues(Bi, m).astype(np.float64)
        want = np.mod(np.rint(ra @ rb).astype(np.int64), m)
        assert np.array_equal(R[l].T.astype(np.int64), want), f"modulus {m}"


@pytest.mark.slow
def test_one_limb_16384_sampled_and_accurate(gpu_lib):
    """m = n = k = 16384 with 18 moduli of the one-limb list (capacities
    50 / 50): sampled outputs bit for bit, and the normalized error of a
    sample within 2^-50."""
    import torch
    N = 16384
    A, B = dgemm_inputs(N, N, N, 0.5, SEED + 8)
    rng = np.random.default_rng(3)
    rows = np.concatenate([[0, N - 1], np.sort(rng.choice(N, 8, replace=False))])
    cols = np.concatenate([[0, N - 1], np.sort(rng.choice(N, 8, replace=False))])
    announce(f"one-limb dgemm {N}^3 L=18, sampled")
    Ad, Bd = dev_cm(A), dev_cm(B)
    Cd = gpu_lib.dgemm(Ad, Bd, 18)
    assert bool(torch.isfinite(Cd).all())
    C = to_np(Cd[torch.as_tensor(rows, device="cuda")][:, torch.as_tensor(cols, device="cuda")])
    del Ad, Bd, Cd
    torch.cuda.empty_cache()
    want = o.dgemm_one_limb(A, B, 18, rows=rows, cols=cols)
    assert (want["cA"], want["cB"]) == (50, 50)
    assert bits_equal(C, want["C"])
    err = o.normalized_errors_block(C[:4, :4], A, B, rows[:4], cols[:4]).max()
    assert err <= 2.0 ** -50


@pytest.fixture
def heads_setting(gpu_lib):
    yield
    gpu_lib.ozfp4_set_one_limb_moduli(0)


@pytest.mark.parametrize("h,m,n,k,L", [
    (2, 131, 67, 129, 12), (3, 300, 300, 200, 19), (4, 200, 130, 333, 21),
    (5, 1000, 200, 300, 21), (5, 33, 97, 64, 4), (5, 64, 64, 500, 5), (5, 256, 256, 1000, 27)])
def test_heads_dgemm_bit_exact(gpu_lib, heads_setting, h, m, n, k, L):
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 20 + h + m)
    want = o.dgemm_one_limb(A, B, L, heads=h)["C"]
    announce(f"dgemm with {h} one-limb heads m={m} n={n} k={k} L={L}")
    assert gpu_lib.ozfp4_set_one_limb_moduli(h) == gpu_lib.OZFP4_OK
    C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), L))
    assert bits_equal(C, want)


def test_heads_residues_bit_exact(gpu_lib, heads_setting):
    m, n, k, L, h = 300, 300, 200, 21, 5
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 30)
    res = o.dgemm_one_limb(A, B, L, heads=h)
    announce(f"residues with {h} one-limb heads m={m} n={n} k={k} L={L}")
    assert gpu_lib.ozfp4_set_one_limb_moduli(h) == gpu_lib.OZFP4_OK
    R = to_np(gpu_lib.residues(dev_cm(A), dev_cm(B), L))
    for l in range(L):
        assert np.array_equal(R[l].T.astype(np.int64), res["r"][l]), f"modulus {res['moduli'][l]}"


def test_heads_same_c_as_the_greedy_lists(gpu_lib, heads_setting):
    """At k = 4096 the 21-moduli lists with 5 and 4 heads have the
    capacities of the greedy 18 (52 / 52) and 19 (53 / 53): the library's C
    is the same bit for bit, and the oracle's."""
    m, n, k = 512, 512, 4096
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 31)
    Ad, Bd = dev_cm(A), dev_cm(B)
    announce("dgemm with 5 / 4 heads and 21 moduli against the greedy 18 / 19")
    gpu_lib.ozfp4_set_one_limb_moduli(0)     # the greedy lists for the reference
    g18 = to_np(gpu_lib.dgemm(Ad, Bd, 18))
    g19 = to_np(gpu_lib.dgemm(Ad, Bd, 19))
    c18, c19 = gpu_lib.ozfp4_capacity(k, 18), gpu_lib.ozfp4_capacity(k, 19)
    gpu_lib.ozfp4_set_one_limb_moduli(5)
    assert gpu_lib.ozfp4_capacity(k, 21) == c18
    h5 = to_np(gpu_lib.dgemm(Ad, Bd, 21))
    gpu_lib.ozfp4_set_one_limb_moduli(4)
    assert gpu_lib.ozfp4_capacity(k, 21) == c19
    h4 = to_np(gpu_lib.dgemm(Ad, Bd, 21))
    gpu_lib.ozfp4_set_one_limb_moduli(0)
    assert bits_equal(h5, g18) and bits_equal(h4, g19)
    assert not bits_equal(g18, g19)
    rows, cols = np.arange(0, m, 97), np.arange(0, n, 131)
    assert bits_equal(h5[np.ix_(rows, cols)], o.dgemm(A, B, 18, rows=rows, cols=cols)["C"])


def test_heads_sgemm_bit_exact(gpu_lib, heads_setting):
    A, B = dgemm_inputs(131, 67, 129, 2.0, SEED + 32)
    A, B = A.astype(np.float32), B.astype(np.float32)
    want = o.sgemm_one_limb(A, B, 13, heads=5)["C"]
    announce("sgemm with 5 one-limb heads, 13 moduli")
    assert gpu_lib.ozfp4_set_one_limb_moduli(5) == gpu_lib.OZFP4_OK
    C = to_np(gpu_lib.sgemm(dev_cm(A), dev_cm(B), 13))
    assert np.array_equal(C.view(np.uint32), want.view(np.uint32))


def test_three_heads_sgemm_same_c_as_greedy(gpu_lib, heads_setting):
    """Three heads with 11 moduli reach the FP32 emulation's 24-bit
    capacities like the 10 greedy moduli, so C is the greedy list's bit for
    bit (34 limb products instead of 39), over several tiles with ragged
    tails; both equal the oracle's."""
    m, n, k = 300, 260, 700
    A, B = dgemm_inputs(m, n, k, 2.0, SEED + 33)
    A, B = A.astype(np.float32), B.astype(np.float32)
    Ad, Bd = dev_cm(A), dev_cm(B)
    gpu_lib.ozfp4_set_one_limb_moduli(0)
    assert gpu_lib.ozfp4_sgemm_capacity(k, 10) == (24, 24)
    announce("sgemm, 10 greedy moduli, then 3 one-limb heads with 11 moduli")
    greedy = to_np(gpu_lib.sgemm(Ad, Bd, 10))
    assert gpu_lib.ozfp4_set_one_limb_moduli(3) == gpu_lib.OZFP4_OK
    assert gpu_lib.ozfp4_sgemm_capacity(k, 11) == (24, 24)
    heads = to_np(gpu_lib.sgemm(Ad, Bd, 11))
    want = o.sgemm_one_limb(A, B, 11, heads=3)["C"]
    assert np.array_equal(heads.view(np.uint32), want.view(np.uint32))
    assert np.array_equal(greedy.view(np.uint32), heads.view(np.uint32))

