"""GPU parity of Ozaki scheme I on FP4 limbs (ozfp4_dgemm_ozi, Sec. IV)
against the CPU oracle, every comparison exact: limb planes byte for byte,
the GEMM's partial sums and C bit for bit. Also the cross-check the paper
states (Sec. VII-A): with 53-bit capacities on both sides, scheme I and
scheme II give bitwise the same C, here both on the GPU."""

import numpy as np
import pytest

import oracle as o
from gpu_util import _code_lut, announce, bits_equal, dev_cm, to_np, unpack_planes
from paper_2608_06812_amd.workloads import dgemm_inputs, paper_law_inputs

pytestmark = pytest.mark.gpu

SEED = 20261102

# (m, n, k, p): several tiles, ragged tails, degenerate sizes, limb counts
# that fill one to five blocks of three
SHAPES = [
    (256, 256, 256, 15),
    (131, 67, 129, 15),
    (1, 1, 1, 15),
    (1, 300, 77, 15),
    (300, 1, 200, 15),
    (200, 130, 333, 15),
    (64, 64, 1000, 15),
    (131, 67, 129, 7),
    (64, 40, 300, 1),
    (100, 90, 200, 4),
    (33, 97, 64, 14),
]


def _codes(limbs, nplanes, rows_pad, k_pad):
    vec = np.vectorize(lambda c: _code_lut[int(c)], otypes=[np.uint8])
    out = np.zeros((nplanes, rows_pad, k_pad), dtype=np.uint8)
    lines, k = limbs[0].shape
    for i, a in enumerate(limbs):
        out[i, :lines, :k] = vec(a)
    return out


def _block_partials(a, b, nblk):
    """H_h = sum_{I + J = h} sum_{i', j' < 3} 13^(i'+j') <a_{3I+i'}, b_{3J+j'}>
    from the oracle's limbs (limbs at or above p are zero)."""
    zero_a, zero_b = np.zeros_like(a[0]), np.zeros_like(b[0])
    a = list(a) + [zero_a] * (3 * nblk - len(a))
    b = list(b) + [zero_b] * (3 * nblk - len(b))
    H = []
    for h in range(2 * nblk - 1):
        acc = np.zeros((a[0].shape[0], b[0].shape[1]), dtype=object)
        for I in range(nblk):
            J = h - I
            if not 0 <= J < nblk:
                continue
            for i2 in range(3):
                for j2 in range(3):
                    prod = a[3 * I + i2].astype(np.float64) @ b[3 * J + j2].astype(np.float64)
                    acc = acc + np.rint(prod).astype(np.int64).astype(object) * 13 ** (i2 + j2)
        H.append(acc)
    return H


@pytest.mark.parametrize("m,n,k,p", [(131, 67, 129, 15), (33, 97, 64, 7), (64, 40, 300, 4),
                                     (40, 20, 90, 1)])
def test_ozi_limb_planes_byte_exact(gpu_lib, m, n, k, p):
    A, B = dgemm_inputs(m, n, k, 1.0, SEED)
    res = o.dgemm_ozi(A, B, p)
    _, nplanes, _ = gpu_lib.ozfp4_ozi_config(p)
    announce(f"ozi limb_planes m={m} n={n} k={k} p={p}")
    pa, pb = gpu_lib.ozi_limb_planes(dev_cm(A), dev_cm(B), p)
    ra, kp, _ = gpu_lib.ozfp4_plane_layout(m, k)
    rbp, _, _ = gpu_lib.ozfp4_plane_layout(n, k)
    assert np.array_equal(unpack_planes(to_np(pa), ra, kp), _codes(res["a"], nplanes, ra, kp))
    assert np.array_equal(unpack_planes(to_np(pb), rbp, kp),
                          _codes([x.T for x in res["b"]], nplanes, rbp, kp))


@pytest.mark.parametrize("m,n,k,p", [(131, 67, 129, 15), (200, 130, 333, 15), (64, 40, 300, 7),
                                     (100, 90, 200, 4)])
def test_ozi_partials_exact(gpu_lib, m, n, k, p):
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 1)
    res = o.dgemm_ozi(A, B, p)
    _, _, ng = gpu_lib.ozfp4_ozi_config(p)
    announce(f"ozi partials m={m} n={n} k={k} p={p}")
    H = to_np(gpu_lib.ozi_partials(dev_cm(A), dev_cm(B), p))
    want = _block_partials(res["a"], res["b"], (p + 2) // 3)
    assert len(want) == ng
    total = np.zeros((m, n), dtype=object)
    for h in range(ng):
        assert np.array_equal(H[h].T.astype(object), want[h]), f"anti-diagonal {h}"
        total = total + H[h].T.astype(object) * 2197 ** h
    assert np.all(total == res["x"])


@pytest.mark.parametrize("m,n,k,p", SHAPES)
def test_ozi_dgemm_bit_exact(gpu_lib, m, n, k, p):
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 2)
    want = o.dgemm_ozi(A, B, p)["C"]
    announce(f"ozi dgemm m={m} n={n} k={k} p={p}")
    C = to_np(gpu_lib.dgemm_ozi(dev_cm(A), dev_cm(B), p))
    assert bits_equal(C, want)


@pytest.mark.parametrize("phi", [0, 1, 8])
def test_ozi_paper_law_inputs(gpu_lib, phi):
    A, B = paper_law_inputs(128, 96, 512, phi, SEED + 3)
    want = o.dgemm_ozi(A, B, 15)["C"]
    announce(f"ozi dgemm paper law phi={phi}")
    C = to_np(gpu_lib.dgemm_ozi(dev_cm(A), dev_cm(B), 15))
    assert bits_equal(C, want)


def test_ozi_edge_values(gpu_lib):
    """Zero lines, subnormal and huge values, exact cancellation."""
    rng = np.random.default_rng(SEED + 4)
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
    want = o.dgemm_ozi(A, B, 15)["C"]
    announce("ozi dgemm edge values")
    C = to_np(gpu_lib.dgemm_ozi(dev_cm(A), dev_cm(B), 15))
    assert bits_equal(C, want)


def test_ozi_k_chunks_at_largest_limbs(gpu_lib):
    """k = 40000 spans three accumulation chunks. Every converted value is
    x = sum_{i<14} 8 13^i + 13^14 (fourteen limbs of 8), the largest limbs
    greedy digits take, so one FP32 accumulation over all of k would exceed
    2^22 and round; the chunked partial sums must stay exact."""
    x = sum(8 * 13 ** i for i in range(14)) + 13 ** 14
    assert 2 ** 52 <= x < 2 ** 53 and o.limb_decompose(x, 15) == [8] * 14 + [1]
    m, n, k = 40, 24, 40000
    A = np.full((m, k), float(x))
    B = np.full((k, n), float(x))
    A[1, :] = -float(x)
    B[:, 2] = -float(x)
    A[3, 1::2] = -float(x)
    res = o.dgemm_ozi(A, B, 15)
    assert np.array_equal(res["Ai"], A.astype(np.int64))
    announce("ozi partials k=40000 largest limbs")
    H = to_np(gpu_lib.ozi_partials(dev_cm(A), dev_cm(B), 15))
    total = np.zeros((m, n), dtype=object)
    for h in range(H.shape[0]):
        total = total + H[h].T.astype(object) * 2197 ** h
    assert np.all(total == res["x"])
    announce("ozi dgemm k=40000 largest limbs")
    C = to_np(gpu_lib.dgemm_ozi(dev_cm(A), dev_cm(B), 15))
    assert bits_equal(C, res["C"])


@pytest.mark.parametrize("m,n,k,phi", [(256, 256, 256, 0.5), (300, 170, 700, 2.0),
                                       (129, 257, 1000, 8.0), (1, 77, 4096, 1.0)])
def test_schemes_agree_bitwise_on_gpu(gpu_lib, m, n, k, phi):
    """Sec. VII-A: scheme I (15 limbs) and scheme II (19 moduli, 53-bit
    capacities) give bitwise the same C; both GPU paths, plus the oracle."""
    assert o.capacity_bits(k, o.select_moduli(19)) == (53, 53)
    A, B = dgemm_inputs(m, n, k, phi, SEED + 5)
    Ad, Bd = dev_cm(A), dev_cm(B)
    announce(f"ozi vs ozii m={m} n={n} k={k}")
    C1 = to_np(gpu_lib.dgemm_ozi(Ad, Bd, 15))
    C2 = to_np(gpu_lib.dgemm(Ad, Bd, 19))
    assert bits_equal(C1, C2)
    rows = np.unique(np.linspace(0, m - 1, 5).astype(int))
    cols = np.unique(np.linspace(0, n - 1, 5).astype(int))
    assert bits_equal(C1[np.ix_(rows, cols)], o.dgemm_ozi(A, B, 15, rows=rows, cols=cols)["C"])


@pytest.mark.slow
def test_ozi_16384_sampled_and_equal_to_ozii(gpu_lib):
    """m = n = k = 16384 in the benchmark's configuration: sampled outputs
    equal the oracle's bit for bit, and the whole C equals scheme II's
    (19 moduli) bit for bit."""
    import torch
    N = 16384
    A, B = dgemm_inputs(N, N, N, 0.5, SEED + 6)
    rows = np.array([0, 1, 4097, 9000, N - 1])
    cols = np.array([0, 2, 8191, 12345, N - 1])
    Ad, Bd = dev_cm(A), dev_cm(B)
    announce("ozi dgemm 16384^3")
    C1 = gpu_lib.dgemm_ozi(Ad, Bd, 15)
    announce("ozii dgemm 16384^3 L=19")
    C2 = gpu_lib.dgemm(Ad, Bd, 19)
    assert torch.equal(C1.view(torch.int64), C2.view(torch.int64))
    sub = to_np(C1[torch.as_tensor(rows, device="cuda")][:, torch.as_tensor(cols, device="cuda")])
    del C1, C2
    want = o.dgemm_ozi(A, B, 15, rows=rows, cols=cols)["C"]
    assert bits_equal(sub, want)


@pytest.mark.slow
def test_ozi_at_the_largest_k_with_largest_limbs(gpu_lib):
    """k = 131072 (OZFP4_MAX_K, eight accumulation chunks of 16384) with
    every converted value at the largest greedy limbs (fourteen limbs of 8,
    then 1): the int64 partial sums reach their largest magnitudes, and the
    partial sums and C stay exact."""
    x = sum(8 * 13 ** i for i in range(14)) + 13 ** 14
    m, n, k = 24, 16, gpu_lib.OZFP4_MAX_K
    A = np.full((m, k), float(x))
    B = np.full((k, n), float(x))
    A[1, :] = -float(x)
    B[:, 2] = -float(x)
    A[3, 1::2] = -float(x)
    res = o.dgemm_ozi(A, B, 15)
    announce(f"ozi partials and dgemm k={k} largest limbs")
    H = to_np(gpu_lib.ozi_partials(dev_cm(A), dev_cm(B), 15))
    total = np.zeros((m, n), dtype=object)
    for h in range(H.shape[0]):
        total = total + H[h].T.astype(object) * 2197 ** h
    assert np.all(total == res["x"])
    C = to_np(gpu_lib.dgemm_ozi(dev_cm(A), dev_cm(B), 15))
    assert bits_equal(C, res["C"])
