"""GPU parity on shapes whose padded tile grid has a multiple of 8 tiles per
modulus. Such grids take the branch of the GEMMs' block-to-tile mapping
that every large workload takes (XCD x gets the x-th eighth of the tile
grid of every modulus in turn); the small ragged shapes of the other tests
have 2 or 4 tiles per modulus and take the other branch. Every output is
compared with the oracle element by element: C bit for bit, residues
exactly.

The residue GEMM's block tile is 256 rows of A by 128 columns of B, and
both operands are padded to 256 lines, so m = n = 300 gives 2 x 4 = 8
tiles, m = 1000, n = 200 gives 4 x 2 = 8 and m = 1024, n = 512 gives
4 x 4 = 16.

At the benchmark workload (m = n = k = 16384, 18 moduli; 64 x 128 = 8192
tiles per modulus), every residue of every modulus is compared with the
definition (A~ B~) mod m formed from the oracle's converted integers:
exactly on the CPU for a quarter of the columns (16 slices of 256 columns
spread over the output, which meet every tile row, so every XCD's share),
and for all 2^28 elements per modulus with the vendor's FP64 matrix
product (torch.matmul, not this library) as the multiplication primitive.
Both are exact: every sum of products of residues is an integer below
168^2 k < 2^53."""

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, bits_equal, dev_cm, to_np
from oracle.sgemm_fp4 import sgemm as oracle_sgemm
from paper_2608_06812_amd.workloads import dgemm_inputs

pytestmark = pytest.mark.gpu

SEED = 20261212


def _tiles(m, n):
    pad = lambda v: (v + 255) // 256 * 256
    return (pad(m) // 256) * (pad(n) // 128)


# (m, n, k, L, cmax, karatsuba)
CASES = [
    (300, 300, 400, 18, 53, False),
    (1000, 200, 300, 18, 53, False),
    (1024, 512, 200, 18, 53, False),
    (512, 512, 256, 14, 53, False),
    (300, 300, 333, 18, 53, True),     # Karatsuba route
    (1000, 200, 129, 19, 53, True),
    (300, 300, 200, 23, 63, False),    # wide-range extension (c up to 63)
    (1024, 512, 131, 27, 63, False),
]


@pytest.mark.parametrize("m,n,k,L,cmax,kar", CASES)
def test_dgemm_full_output_on_the_xcd_share_mapping(gpu_lib, m, n, k, L, cmax, kar):
    assert _tiles(m, n) % 8 == 0
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + m + 7 * n + 13 * k)
    want = o.dgemm(A, B, L, cmax=cmax)
    announce(f"tile mapping dgemm m={m} n={n} k={k} L={L} cmax={cmax} karatsuba={kar}")
    try:
        gpu_lib.ozfp4_set_max_capacity(cmax)
        gpu_lib.ozfp4_set_karatsuba(kar)
        Ad, Bd = dev_cm(A), dev_cm(B)
        R = to_np(gpu_lib.residues(Ad, Bd, L))
        C = to_np(gpu_lib.dgemm(Ad, Bd, L))
    finally:
        gpu_lib.ozfp4_set_karatsuba(False)
        gpu_lib.ozfp4_set_max_capacity(53)
    for l in range(L):
        assert np.array_equal(R[l].T.astype(np.int64), want["r"][l]), f"modulus {want['moduli'][l]}"
    assert bits_equal(C, want["C"])


def test_sgemm_full_output_on_the_xcd_share_mapping(gpu_lib):
    import torch
    m, n, k, L = 300, 300, 500, 10
    assert _tiles(m, n) % 8 == 0
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 1)
    A, B = A.astype(np.float32), B.astype(np.float32)
    want = oracle_sgemm(A, B, L)["C"]
    announce(f"tile mapping sgemm m={m} n={n} k={k} L={L}")
    Ad = torch.from_numpy(np.ascontiguousarray(A.T)).cuda().t()
    Bd = torch.from_numpy(np.ascontiguousarray(B.T)).cuda().t()
    C = gpu_lib.sgemm(Ad, Bd, L).cpu().numpy()
    assert np.array_equal(C.view(np.uint32), want.view(np.uint32))


def test_residues_4096_every_modulus_full(gpu_lib):
    """m = n = k = 4096 with 18 moduli (16 x 32 = 512 tiles per modulus):
    all 2^24 residues of every modulus against ((A~ mod m)(B~ mod m)) mod m
    from the oracle's converted integers, one exact CPU FP64 product per
    modulus."""
    N, L = 4096, 18
    A, B = dgemm_inputs(N, N, N, 0.5, SEED + 2)
    moduli = o.select_moduli(L)
    cA, cB = o.capacity_bits(N, moduli)
    Ai = o.to_integers(A, o.shift_exponents(A, axis=1, c=cA), axis=1)
    Bi = o.to_integers(B, o.shift_exponents(B, axis=0, c=cB), axis=0)
    announce("residues 4096^3 L=18, every modulus in full")
    R = to_np(gpu_lib.residues(dev_cm(A), dev_cm(B), L))
    assert 168.0 ** 2 * N < 2.0 ** 53
    for l, m in enumerate(moduli):
        ra = o.residues(Ai, m).astype(np.float64)
        rb = o.residues(Bi, m).astype(np.float64)
        want = np.mod(np.rint(ra @ rb).astype(np.int64), m)
        assert np.array_equal(R[l].T.astype(np.int64), want), f"modulus {m}"


@pytest.fixture(scope="module")
def bench_residues(gpu_lib):
    """The library's residues at the benchmark workload (host copy, one
    (n, m) uint8 matrix per modulus) and the oracle's converted integers."""
    import torch
    N, L = 16384, 18
    A, B = dgemm_inputs(N, N, N, 0.5, SEED + 3)
    moduli = o.select_moduli(L)
    cA, cB = o.capacity_bits(N, moduli)
    Ai = o.to_integers(A, o.shift_exponents(A, axis=1, c=cA), axis=1)
    Bi = o.to_integers(B, o.shift_exponents(B, axis=0, c=cB), axis=0)
    announce("residues 16384^3 L=18 (all moduli)")
    Ad, Bd = dev_cm(A), dev_cm(B)
    del A, B
    R = gpu_lib.residues(Ad, Bd, L)
    got = R.cpu().numpy()
    del R, Ad, Bd
    torch.cuda.empty_cache()
    return {"N": N, "moduli": moduli, "Ai": Ai, "Bi": Bi, "R": got}


def _column_slices(N, count=16, width=256):
    """count slices of width columns, one in each N / count block of columns
    at a varying offset inside it."""
    step = N // count
    starts = [s * step + (s * 37) % (step - width) for s in range(count)]
    return np.concatenate([np.arange(a, a + width) for a in starts])


@pytest.mark.slow
@pytest.mark.parametrize("part", [0, 1, 2])
def test_residues_16384_every_modulus_quarter_columns_cpu(gpu_lib, bench_residues, part):
    """A third of the moduli per test: for each, a quarter of the columns of
    the benchmark output (every row) against the exact CPU product."""
    d = bench_residues
    N, moduli = d["N"], d["moduli"]
    cols = _column_slices(N)
    assert len(cols) == N // 4 and len(np.unique(cols)) == len(cols)
    assert 168.0 ** 2 * N < 2.0 ** 53
    for l in range(part, len(moduli), 3):
        m = moduli[l]
        announce(f"residues 16384^3 modulus {m}: CPU check of {len(cols)} columns")
        ra = o.residues(d["Ai"], m).astype(np.float64)
        rb = o.residues(d["Bi"][:, cols], m).astype(np.float64)
        want = np.mod(np.rint(ra @ rb).astype(np.int64), m)      # (N, len(cols))
        got = d["R"][l][cols, :].T.astype(np.int64)
        assert np.array_equal(got, want), f"modulus {m}"


@pytest.mark.slow
def test_residues_16384_every_modulus_full_vendor_product(gpu_lib, bench_residues):
    """Every one of the 18 x 2^28 residues against (A~ mod m)(B~ mod m) mod m,
    the oracle's residues multiplied by torch.matmul in FP64 on the GPU
    (vendor BLAS, exact here since every partial sum is an integer below
    2^53)."""
    import torch
    d = bench_residues
    N, moduli = d["N"], d["moduli"]
    for l, m in enumerate(moduli):
        announce(f"residues 16384^3 modulus {m}: full check with the vendor FP64 product")
        ra = torch.from_numpy(o.residues(d["Ai"], m).astype(np.float64)).cuda()
        rb = torch.from_numpy(o.residues(d["Bi"], m).astype(np.float64)).cuda()
        prod = torch.matmul(ra, rb)
        del ra, rb
        want = torch.remainder(torch.round(prod).to(torch.int64), m).to(torch.uint8)
        del prod
        got = torch.from_numpy(d["R"][l]).cuda().t()
        assert torch.equal(got, want), f"modulus {m}"
        del want, got
        torch.cuda.empty_cache()
