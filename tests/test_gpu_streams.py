"""The library runs on the caller's stream (ozfp4_set_stream; the torch
helpers pass torch's current stream): work queued on a side stream before a
call is complete before the library reads its inputs, and work queued after
it sees the finished output. A spin kernel delays the producer of the
input on the side stream, so a call issued on any other stream would read
the input before it is written."""

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, bits_equal, dev_cm, to_np
from paper_2608_06812_amd.workloads import dgemm_inputs, int8_inputs

pytestmark = pytest.mark.gpu

SEED = 20261203
SPIN_CYCLES = 20_000_000   # about 10 ms of a spinning kernel


def test_dgemm_on_a_side_stream(gpu_lib):
    import torch
    m, n, k = 200, 150, 300
    A, B = dgemm_inputs(m, n, k, 0.5, SEED)
    want = o.dgemm(A, B, 19)["C"]
    Ad, Bd = dev_cm(A), dev_cm(B)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    announce("dgemm on a side stream after a spin kernel")
    with torch.cuda.stream(side):
        torch.cuda._sleep(SPIN_CYCLES)
        A2 = Ad * 2.0                 # exact; written only after the spin
        C = gpu_lib.dgemm(A2, Bd, 19)
        D = C * 0.5                   # exact: fl(2 A B) = 2 fl(A B) here
    torch.cuda.synchronize()
    assert bits_equal(to_np(D), want)


def test_igemm_s8_on_a_side_stream(gpu_lib):
    """ozfp4_igemm_s8 is asynchronous: ordering on the side stream is all
    that makes its inputs ready and its output complete."""
    import torch
    m, n, k = 256, 192, 640
    A, B = int8_inputs(m, n, k, SEED + 1)
    want = (A.astype(np.int64) @ B.astype(np.int64)).astype(np.int32)
    Ad = torch.from_numpy(np.ascontiguousarray(A.T)).cuda().t()
    Bd = torch.from_numpy(np.ascontiguousarray(B.T)).cuda().t()
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    announce("igemm_s8 on a side stream after a spin kernel")
    with torch.cuda.stream(side):
        torch.cuda._sleep(SPIN_CYCLES)
        A2 = Ad.clone()
        C = gpu_lib.igemm_s8(A2, Bd)
        D = C.clone()
    torch.cuda.synchronize()
    assert np.array_equal(D.cpu().numpy(), want)


def test_finalize_then_reuse(gpu_lib):
    """ozfp4_finalize releases the workspace and tables of every device; the
    next call sets them up again and gives the same bits."""
    import torch
    m, n, k = 90, 70, 200
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 2)
    A8, B8 = int8_inputs(m, n, k, SEED + 3)
    Ad, Bd = dev_cm(A), dev_cm(B)
    A8d = torch.from_numpy(np.ascontiguousarray(A8.T)).cuda().t()
    B8d = torch.from_numpy(np.ascontiguousarray(B8.T)).cuda().t()
    announce("dgemm, finalize, dgemm and igemm_s8 again")
    C1 = to_np(gpu_lib.dgemm(Ad, Bd, 19))
    assert gpu_lib.ozfp4_finalize() == gpu_lib.OZFP4_OK
    C2 = to_np(gpu_lib.dgemm(Ad, Bd, 19))
    assert gpu_lib.ozfp4_finalize() == gpu_lib.OZFP4_OK
    C3 = gpu_lib.igemm_s8(A8d, B8d).cpu().numpy()
    assert bits_equal(C1, C2) and bits_equal(C1, o.dgemm(A, B, 19)["C"])
    assert np.array_equal(C3, o.igemm_s8(A8, B8))


def test_workspace_allocation_failure_is_reported_and_recovered(gpu_lib):
    """Sizes that pass the argument checks but need a workspace far beyond
    the device's memory return OZFP4_ENOMEM before any kernel runs (the
    small buffers passed are never read); the next call of normal size
    allocates again and is exact."""
    import torch
    total = torch.cuda.get_device_properties(0).total_memory
    big, kk = 1 << 20, 1 << 16          # dgemm: m = n = 2^20, k = 1
    m8 = 1 << 24                        # igemm_s8: m = n = 2^24, k = 2^16
    dgemm_ws = big * big * 19           # residue bytes alone
    igemm_ws = 2 * 3 * m8 * kk // 2     # limb planes of A and B
    if min(dgemm_ws, igemm_ws) < 2 * total:
        pytest.skip("device memory too large for a certain allocation failure")
    dummy = torch.zeros(16, dtype=torch.float64, device="cuda")
    dummy8 = torch.zeros(16, dtype=torch.int8, device="cuda")
    out32 = torch.zeros(16, dtype=torch.int32, device="cuda")
    announce("dgemm and igemm_s8 with a workspace beyond the device: ENOMEM")
    p = dummy.data_ptr()
    assert gpu_lib.ozfp4_dgemm(big, big, 1, p, big, p, 1, p, big, 19) == gpu_lib.OZFP4_ENOMEM
    assert gpu_lib.ozfp4_igemm_s8(m8, m8, kk, dummy8.data_ptr(), m8, dummy8.data_ptr(), kk,
                                  out32.data_ptr(), m8) == gpu_lib.OZFP4_ENOMEM
    torch.cuda.synchronize()
    assert float(dummy.abs().sum()) == 0.0 and int(out32.abs().sum()) == 0
    m, n, k = 60, 50, 100
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 4)
    announce("dgemm of normal size after ENOMEM")
    C = to_np(gpu_lib.dgemm(dev_cm(A), dev_cm(B), 19))
    assert bits_equal(C, o.dgemm(A, B, 19)["C"])


def test_stage_times_after_finalize(gpu_lib):
    """A profiled asynchronous call whose events were released by
    ozfp4_finalize leaves no stage times behind (and no stale events)."""
    import torch
    A8, B8 = int8_inputs(64, 64, 128, SEED + 5)
    Ad = torch.from_numpy(np.ascontiguousarray(A8.T)).cuda().t()
    Bd = torch.from_numpy(np.ascontiguousarray(B8.T)).cuda().t()
    announce("profiled igemm_s8, finalize, stage times")
    gpu_lib.ozfp4_profile(True)
    try:
        gpu_lib.igemm_s8(Ad, Bd)
        torch.cuda.synchronize()
        assert gpu_lib.ozfp4_finalize() == gpu_lib.OZFP4_OK
        assert gpu_lib.ozfp4_stage_times() == []
        C = gpu_lib.igemm_s8(Ad, Bd).cpu().numpy()
        assert len(gpu_lib.ozfp4_stage_times()) == 3
    finally:
        gpu_lib.ozfp4_profile(False)
    assert np.array_equal(C, o.igemm_s8(A8, B8))


def test_stage_times_of_pending_call_survive_a_hook(gpu_lib):
    """A profiled asynchronous igemm_s8 leaves its stage events pending; a
    parity hook that runs next records over the same events (ozfp4_scales
    records two of them). The pending times must be read before that: the
    three igemm stages come back non-negative, and a profiled dgemm after
    them reports its own five."""
    import torch
    A8, B8 = int8_inputs(512, 512, 4096, SEED + 6)
    Ad = torch.from_numpy(np.ascontiguousarray(A8.T)).cuda().t()
    Bd = torch.from_numpy(np.ascontiguousarray(B8.T)).cuda().t()
    A, B = dgemm_inputs(300, 300, 300, 0.5, SEED + 7)
    Ag, Bg = dev_cm(A), dev_cm(B)
    announce("profiled igemm_s8, then ozfp4_scales, then stage times")
    gpu_lib.ozfp4_profile(True)
    try:
        gpu_lib.igemm_s8(Ad, Bd)
        gpu_lib.scales(Ag, Bg, 18)
        st = gpu_lib.ozfp4_stage_times()
        assert len(st) == 3 and all(x >= 0.0 for x in st), st
        assert st[2] > 0.0
        gpu_lib.igemm_s8(Ad, Bd)
        gpu_lib.limb_planes(Ag, Bg, 18)
        st2 = gpu_lib.ozfp4_stage_times()
        assert len(st2) == 3 and all(x >= 0.0 for x in st2), st2
        gpu_lib.dgemm(Ag, Bg, 18)
        st3 = gpu_lib.ozfp4_stage_times()
        assert len(st3) == 5 and all(x >= 0.0 for x in st3), st3
    finally:
        gpu_lib.ozfp4_profile(False)
