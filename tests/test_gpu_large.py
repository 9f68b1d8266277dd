"""GPU checks of outputs too large for one kernel launch (a launch holds
fewer than 2^32 work-items): the zero fill of k = 0, the CRT and the column
maxima of B are split over several launches or stride over a bounded grid.

With k = 1 and inputs +-(1 or 1.5) 2^e, every converted value is exact at
the two-moduli capacities (7 and 6 bits), so C_ij = A_i0 B_0j exactly; the
reference is torch's outer product on the GPU, compared bit for bit. The
binades vary per line, so a line whose maximum or shift went missing would
show up as a wrong value."""

import numpy as np
import pytest

from gpu_util import announce

pytestmark = pytest.mark.gpu

SEED = 20261202


def _two_bit_values(n, seed):
    rng = np.random.default_rng(seed)
    mant = np.where(rng.random(n) < 0.5, 1.0, 1.5)
    sign = np.where(rng.random(n) < 0.5, -1.0, 1.0)
    return sign * mant * np.exp2(rng.integers(-20, 21, size=n))


def _col(v, dtype):
    import torch
    return torch.as_tensor(v, dtype=dtype, device="cuda").reshape(-1, 1)


def _row(v, dtype):
    import torch
    return torch.as_tensor(v, dtype=dtype, device="cuda").reshape(1, -1)


def _cm_full(m, n, value, dtype):
    import torch
    return torch.full((n, m), value, dtype=dtype, device="cuda").t()


def _all_zero_bits(C, int_dtype):
    import torch
    v = C.view(int_dtype)
    return int(torch.amax(v)) == 0 and int(torch.amin(v)) == 0


def _free():
    import torch
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_k_zero_fill_beyond_one_launch(gpu_lib):
    """k = 0 writes +0 to every element of a C with m n > 2^32."""
    import torch
    m, n = 65536, 65537
    assert m * n > 2 ** 32
    _free()
    A = torch.empty((m, 0), dtype=torch.float64, device="cuda")
    B = torch.empty((0, n), dtype=torch.float64, device="cuda")
    C = _cm_full(m, n, 7.0, torch.float64)
    announce(f"dgemm k=0 m={m} n={n}")
    gpu_lib.dgemm(A, B, 19, out=C)
    assert _all_zero_bits(C, torch.int64)
    del C
    _free()
    C = _cm_full(m, n, 7.0, torch.float32)
    announce(f"sgemm k=0 m={m} n={n}")
    gpu_lib.sgemm(A.float(), B.float(), 10, out=C)
    assert _all_zero_bits(C, torch.int32)
    del C
    _free()
    C = _cm_full(m, n, 7, torch.int32)
    announce(f"igemm_s8 k=0 m={m} n={n}")
    gpu_lib.igemm_s8(A.to(torch.int8), B.to(torch.int8), out=C)
    torch.cuda.synchronize()
    assert _all_zero_bits(C, torch.int32)
    del C
    _free()


@pytest.mark.parametrize("fp32", [False, True])
def test_crt_beyond_one_launch(gpu_lib, fp32):
    """m = n = 65600: the CRT's ceil(m/4) n threads exceed 2^30, so it takes
    two launches; every output equals the exact product."""
    import torch
    m = n = 65600
    assert (m // 4) * n > 2 ** 30
    dt = torch.float32 if fp32 else torch.float64
    it = torch.int32 if fp32 else torch.int64
    a = _two_bit_values(m, SEED)
    b = _two_bit_values(n, SEED + 1)
    _free()
    A, B = _col(a, dt), _row(b, dt)
    announce(f"{'sgemm' if fp32 else 'dgemm'} k=1 m=n={m} L=2 (CRT over two launches)")
    C = gpu_lib.sgemm(A, B, 2) if fp32 else gpu_lib.dgemm(A, B, 2)
    want = torch.outer(A[:, 0], B[0, :])
    assert torch.equal(C.view(it), want.view(it))
    del C, want
    _free()


@pytest.mark.parametrize("fp32", [False, True])
def test_column_maxima_beyond_one_launch(gpu_lib, fp32):
    """n = 2^24 + 4096 columns of B, one wave each: more than one launch
    holds, so the column maxima take two launches."""
    import torch
    m, n = 3, 2 ** 24 + 4096
    dt = torch.float32 if fp32 else torch.float64
    it = torch.int32 if fp32 else torch.int64
    a = _two_bit_values(m, SEED + 2)
    b = _two_bit_values(n, SEED + 3)
    _free()
    A, B = _col(a, dt), _row(b, dt)
    announce(f"{'sgemm' if fp32 else 'dgemm'} k=1 m={m} n={n} L=2 (column maxima over two launches)")
    C = gpu_lib.sgemm(A, B, 2) if fp32 else gpu_lib.dgemm(A, B, 2)
    want = torch.outer(A[:, 0], B[0, :])
    assert torch.equal(C.view(it), want.view(it))
    del C, want
    _free()
