"""GPU parity of the bit-exact INT8 x INT8 -> INT32 product on FP4 limbs
(Sec. III) against the integer oracle."""

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, dev_cm, to_np
from paper_2608_06812_amd.workloads import int8_inputs

pytestmark = pytest.mark.gpu

SEED = 20260811


@pytest.mark.parametrize("m,n,k", [
    (128, 64, 128), (1, 1, 1), (131, 67, 129), (300, 200, 1000), (64, 65, 4097), (17, 300, 2),
])
def test_igemm_s8_bit_exact(gpu_lib, m, n, k):
    A, B = int8_inputs(m, n, k, SEED)
    want = o.igemm_s8(A, B)
    announce(f"igemm_s8 m={m} n={n} k={k}")
    C = to_np(gpu_lib.igemm_s8(dev_cm(A), dev_cm(B)))
    assert np.array_equal(C, want)


def test_igemm_s8_extremes_at_the_fp32_limit(gpu_lib):
    """All -128 (the largest limb products) at k = 87381, the FP32-exactness
    limit of one grouped accumulation (the library runs it as two chunks);
    plus mixed signs."""
    k = 87381
    A = np.full((128, k), -128, dtype=np.int8)
    B = np.full((k, 64), -128, dtype=np.int8)
    A[1::2, :] = 127
    B[:, 1::3] = -127
    A[:, -1] = 1
    want = o.igemm_s8(A, B)
    announce(f"igemm_s8 extremes k={k}")
    C = to_np(gpu_lib.igemm_s8(dev_cm(A), dev_cm(B)))
    assert np.array_equal(C, want)


def test_igemm_s8_long_k_chunks_and_wraps(gpu_lib):
    """k = 200000: three accumulation chunks, and with every value -128 the
    exact products reach 2^31.6, so C must wrap modulo 2^32 like INT32
    accumulation; mixed signs and a ragged shape around it."""
    k = 200000
    A = np.full((70, k), -128, dtype=np.int8)
    B = np.full((k, 40), -128, dtype=np.int8)
    A[1::3, :] = 127
    B[:, 2::5] = 3
    A[5, ::7] = -1
    want = o.igemm_s8(A, B)
    assert np.abs(A[:1].astype(np.int64) @ B[:, :1].astype(np.int64)).max() > 2 ** 31
    announce(f"igemm_s8 k={k}")
    C = to_np(gpu_lib.igemm_s8(dev_cm(A), dev_cm(B)))
    assert np.array_equal(C, want)


def test_igemm_s8_k_zero(gpu_lib):
    import torch
    announce("igemm_s8 k=0")
    C = gpu_lib.igemm_s8(dev_cm(np.zeros((4, 0), dtype=np.int8)), dev_cm(np.zeros((0, 3), dtype=np.int8)))
    assert C.shape == (4, 3) and bool(torch.all(C == 0))


@pytest.mark.slow
def test_igemm_s8_8192_full(gpu_lib):
    """The INT8 configuration (8192^3): 48 whole rows and 48 whole columns
    of C against the oracle, and every element of C against the definition
    A B formed by one FP64 product of the int8 inputs, exact here because
    |sum| <= 128^2 8192 = 2^27 < 2^53 (and below 2^31, so nothing wraps)."""
    A, B = int8_inputs(8192, 8192, 8192, SEED + 1)
    announce("igemm_s8 8192^3")
    Cd = gpu_lib.igemm_s8(dev_cm(A), dev_cm(B))
    rng = np.random.default_rng(5)
    rows = np.sort(rng.choice(8192, 48, replace=False))
    cols = np.sort(rng.choice(8192, 48, replace=False))
    import torch
    got_rows = to_np(Cd[torch.as_tensor(rows, device="cuda")])
    got_cols = to_np(Cd[:, torch.as_tensor(cols, device="cuda")])
    assert np.array_equal(got_rows, o.igemm_s8(A[rows], B))
    assert np.array_equal(got_cols, o.igemm_s8(A, B[:, cols]))
    want = np.rint(A.astype(np.float64) @ B.astype(np.float64)).astype(np.int64)
    assert np.abs(want).max() < 2 ** 31
    assert np.array_equal(to_np(Cd).astype(np.int64), want)


def test_igemm_s8_equals_native_int8_matrix_cores(gpu_lib):
    """The FP4-limb product equals the GPU's own INT8 matrix product
    (torch._int_mm, int32 accumulation) bit for bit, including results that
    wrap modulo 2^32."""
    import torch
    A, B = int8_inputs(256, 192, 4096, SEED + 2)
    A[:3, :] = -128
    B[:, :2] = -128
    announce("igemm_s8 against native int8 256x192x4096")
    C = gpu_lib.igemm_s8(dev_cm(A), dev_cm(B))
    native = torch._int_mm(torch.from_numpy(A).cuda(), torch.from_numpy(np.ascontiguousarray(B)).cuda())
    assert torch.equal(C, native)
    assert np.array_equal(to_np(C), o.igemm_s8(A, B))
