"""GPU parity of the FP32 emulation (ozfp4_sgemm): C bit for bit against
the oracle's single binary32 rounding of the exact product of the converted
inputs, on ragged shapes, several moduli counts, FP32 edge values
(subnormals, overflow to inf, cancellation), and sampled outputs of the
16384^3 workload with its accuracy against the exact product."""

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, dev_cm, to_np
from paper_2608_06812_amd.workloads import dgemm_inputs

pytestmark = pytest.mark.gpu

SEED = 20261202

SHAPES = [
    (256, 256, 256, 10),
    (131, 67, 129, 10),
    (1, 1, 1, 10),
    (1, 300, 77, 10),
    (300, 1, 200, 8),
    (200, 130, 333, 12),
    (64, 64, 1000, 10),
    (33, 97, 64, 5),
    (100, 90, 4000, 19),
]


def _f32_inputs(m, n, k, phi, seed):
    A, B = dgemm_inputs(m, n, k, phi, seed)
    return A.astype(np.float32), B.astype(np.float32)


def _same(a, b):
    a = np.ascontiguousarray(a, dtype=np.float32)
    b = np.ascontiguousarray(b, dtype=np.float32)
    return a.shape == b.shape and np.array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("m,n,k,L", SHAPES)
def test_sgemm_bit_exact(gpu_lib, m, n, k, L):
    A, B = _f32_inputs(m, n, k, 0.5, SEED)
    want = o.sgemm(A, B, L)["C"]
    announce(f"sgemm m={m} n={n} k={k} L={L}")
    C = to_np(gpu_lib.sgemm(dev_cm(A), dev_cm(B), L))
    assert _same(C, want)


def test_sgemm_default_moduli_and_wide_exponents(gpu_lib):
    A, B = _f32_inputs(150, 70, 500, 8.0, SEED + 1)
    L = gpu_lib.sgemm_moduli(500)
    assert gpu_lib.ozfp4_sgemm_capacity(500, L) == (24, 24)
    want = o.sgemm(A, B, L)["C"]
    announce(f"sgemm default moduli L={L} phi=8")
    C = to_np(gpu_lib.sgemm(dev_cm(A), dev_cm(B)))
    assert _same(C, want)


def test_sgemm_edge_values(gpu_lib):
    """Zero lines, FP32 subnormals in and out, overflow to inf, exact
    cancellation, and a line of maximal FP32 values."""
    rng = np.random.default_rng(SEED + 2)
    m, n, k = 70, 50, 90
    A = ((rng.random((m, k)) - 0.5) * np.exp2(rng.integers(-30, 30, size=(m, k)))).astype(np.float32)
    B = ((rng.random((k, n)) - 0.5) * np.exp2(rng.integers(-30, 30, size=(k, n)))).astype(np.float32)
    A[0, :] = 0
    B[:, 1] = 0
    A[2, :] = np.float32(1e-39)                    # subnormal inputs
    A[3, :] *= np.float32(1e-30)                   # results below the subnormal range
    A[4, :] = np.float32(3e38)
    B[:, 5] = np.float32(3e38)                     # overflow to +-inf
    A[6, :5] = np.array([1.4e-45, -1.4e-45, 1e-40, 2.5, 0.5], dtype=np.float32)
    A[7, :] = 1
    B[:, 7] = 0
    B[0, 7], B[1, 7] = 1, -1                       # exact cancellation
    A[8, :] = np.finfo(np.float32).max
    want = o.sgemm(A, B, 10)["C"]
    announce("sgemm edge values")
    C = to_np(gpu_lib.sgemm(dev_cm(A), dev_cm(B), 10))
    assert _same(C, want)
    assert np.isinf(C[4, 5])


def test_sgemm_errors_and_empty(gpu_lib):
    import torch
    A, B = _f32_inputs(20, 10, 30, 0.5, SEED + 3)
    A[3, 4] = np.nan
    announce("sgemm non-finite input")
    with pytest.raises(gpu_lib.OzFP4Error) as err:
        gpu_lib.sgemm(dev_cm(A), dev_cm(B), 10)
    assert err.value.code == gpu_lib.OZFP4_ENONFINITE
    announce("sgemm k = 0")
    Z = gpu_lib.sgemm(torch.empty((5, 0), dtype=torch.float32, device="cuda"),
                      torch.empty((0, 3), dtype=torch.float32, device="cuda"), 10)
    assert np.array_equal(to_np(Z).view(np.uint32), np.zeros((5, 3), dtype=np.uint32))


def test_sgemm_ignores_karatsuba_setting(gpu_lib):
    A, B = _f32_inputs(130, 140, 300, 1.0, SEED + 4)
    Ad, Bd = dev_cm(A), dev_cm(B)
    announce("sgemm with the Karatsuba setting on")
    C0 = to_np(gpu_lib.sgemm(Ad, Bd, 12))
    gpu_lib.ozfp4_set_karatsuba(True)
    try:
        C1 = to_np(gpu_lib.sgemm(Ad, Bd, 12))
    finally:
        gpu_lib.ozfp4_set_karatsuba(False)
    assert _same(C0, C1) and _same(C0, o.sgemm(A, B, 12)["C"])


@pytest.mark.slow
def test_sgemm_16384_sampled_and_accuracy(gpu_lib):
    """m = n = k = 16384 with 10 moduli (the benchmark's configuration):
    sampled outputs bit for bit, and the normalized error on a sample within
    2^-22 (native FP32 matrix multiplication's is printed beside it)."""
    import torch
    N = 16384
    A, B = _f32_inputs(N, N, N, 0.5, SEED + 5)
    rows = np.array([0, 1, 4097, 9000, N - 1])
    cols = np.array([0, 2, 8191, 12345, N - 1])
    Ad, Bd = dev_cm(A), dev_cm(B)
    announce("sgemm 16384^3 L=10")
    C = gpu_lib.sgemm(Ad, Bd, 10)
    r = torch.as_tensor(rows, device="cuda")
    c = torch.as_tensor(cols, device="cuda")
    sub = to_np(C[r][:, c])
    assert _same(sub, o.sgemm(A, B, 10, rows=rows, cols=cols)["C"])
    announce("native fp32 matmul 16384^3")
    Cn = to_np(torch.matmul(torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda())[r][:, c])
    A64, B64 = A.astype(np.float64), B.astype(np.float64)
    err = o.normalized_errors_block(sub.astype(np.float64), A64, B64, rows, cols)
    err_n = o.normalized_errors_block(Cn.astype(np.float64), A64, B64, rows, cols)
    announce(f"normalized error: emulated {err.max():.3e}, native {err_n.max():.3e}")
    assert err.max() <= 2.0 ** -22


@pytest.mark.slow
def test_sgemm_at_the_largest_k(gpu_lib):
    """k = 131072 (OZFP4_MAX_K) with the default moduli for 24-bit
    capacities, wide exponents and adversarial all-equal lines: C bit for
    bit against the oracle."""
    import torch
    m, n, k = 40, 24, gpu_lib.OZFP4_MAX_K
    L = gpu_lib.sgemm_moduli(k)
    A, B = dgemm_inputs(m, n, k, 2.0, SEED + 20)
    A, B = A.astype(np.float32), B.astype(np.float32)
    A[0, :] = np.float32(3.0)
    B[:, 0] = np.float32(-5.0)
    want = o.sgemm(A, B, L)["C"]
    announce(f"sgemm k={k} L={L}")
    Ad = torch.from_numpy(np.ascontiguousarray(A.T)).cuda().t()
    Bd = torch.from_numpy(np.ascontiguousarray(B.T)).cuda().t()
    C = gpu_lib.sgemm(Ad, Bd).cpu().numpy()
    assert np.array_equal(C.view(np.uint32), want.view(np.uint32))
