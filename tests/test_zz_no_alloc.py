"""GPU checks of ozfp4_dgemm_noalloc, the entry point that allocates
nothing: through the C ABI, two calls in a row (the second smaller) give C
bit for bit equal to ozfp4_dgemm's on the same inputs and to the oracle's;
the device's free memory does not change across the calls; calls beyond the
fixed scratch or on a device that was not set up are refused before any GPU
work; ozfp4_dgemm still works afterwards; recorded into a graph by stream
capture and replayed several times, with eager work between the replays,
every replay gives the eager result."""

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, bits_equal, dev_cm, to_np
from paper_2608_06812_amd.workloads import dgemm_inputs

pytestmark = pytest.mark.gpu

SEED = 20261220


def _call_noalloc(lib, Ad, Bd, C, L):
    m, k = Ad.shape
    n = Bd.shape[1]
    return lib.ozfp4_dgemm_noalloc(m, n, k, Ad.data_ptr(), Ad.stride(1), Bd.data_ptr(),
                                   Bd.stride(1), C.data_ptr(), C.stride(1), L)


def test_noalloc_matches_dgemm_twice_then_smaller(gpu_lib):
    import torch
    assert gpu_lib.ozfp4_init() == gpu_lib.OZFP4_OK
    # a first tiny call, so that nothing the runtime sets up lazily on a
    # first launch falls inside the measured calls
    A1, B1 = dgemm_inputs(1, 1, 1, 0.5, SEED)
    C1 = torch.zeros((1, 1), dtype=torch.float64, device="cuda")
    gpu_lib.ozfp4_set_stream(torch.cuda.current_stream().cuda_stream)
    assert _call_noalloc(gpu_lib, dev_cm(A1), dev_cm(B1), C1, 14) == gpu_lib.OZFP4_OK
    torch.cuda.synchronize()
    cases = [(700, 500, 900, 18), (300, 200, 100, 14)]
    for m, n, k, L in cases:
        A, B = dgemm_inputs(m, n, k, 0.5, SEED + m)
        Ad, Bd = dev_cm(A), dev_cm(B)
        C = torch.full((n, m), float("nan"), dtype=torch.float64, device="cuda").t()
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        announce(f"dgemm_noalloc m={m} n={n} k={k} L={L}")
        gpu_lib.ozfp4_set_stream(torch.cuda.current_stream().cuda_stream)
        assert _call_noalloc(gpu_lib, Ad, Bd, C, L) == gpu_lib.OZFP4_OK
        torch.cuda.synchronize()
        assert torch.cuda.mem_get_info()[0] == free0      # nothing allocated
        want = to_np(gpu_lib.dgemm(Ad, Bd, L))
        got = to_np(C)
        assert bits_equal(got, want)
        assert bits_equal(got, o.dgemm(A, B, L)["C"])


def test_noalloc_refusals_and_dgemm_after(gpu_lib):
    import torch
    assert gpu_lib.ozfp4_init() == gpu_lib.OZFP4_OK
    A, B = dgemm_inputs(64, 64, 64, 0.5, SEED)
    Ad, Bd = dev_cm(A), dev_cm(B)
    C = torch.zeros((64, 64), dtype=torch.float64, device="cuda").t()
    # 4096^3 with 18 moduli needs about 0.9 GB: beyond the fixed scratch;
    # refused on the host (the pointers are never touched)
    big = 4096
    assert gpu_lib.ozfp4_dgemm_noalloc(big, big, big, Ad.data_ptr(), big, Bd.data_ptr(), big,
                                       C.data_ptr(), big, 18) == gpu_lib.OZFP4_ESCRATCH
    # finalize releases the device set-up: refused until ozfp4_init again
    assert gpu_lib.ozfp4_finalize() == gpu_lib.OZFP4_OK
    assert _call_noalloc(gpu_lib, Ad, Bd, C, 16) == gpu_lib.OZFP4_ESCRATCH
    assert gpu_lib.ozfp4_init() == gpu_lib.OZFP4_OK
    announce("dgemm_noalloc after finalize and init, then dgemm")
    gpu_lib.ozfp4_set_stream(torch.cuda.current_stream().cuda_stream)
    assert _call_noalloc(gpu_lib, Ad, Bd, C, 16) == gpu_lib.OZFP4_OK
    torch.cuda.synchronize()
    want = o.dgemm(A, B, 16)["C"]
    assert bits_equal(to_np(C), want)
    assert bits_equal(to_np(gpu_lib.dgemm(Ad, Bd, 16)), want)


def test_noalloc_captured_graph_replays(gpu_lib):
    """Recorded into a graph by torch's stream capture and replayed three
    times, with the program's own eager work between the replays (C cleared
    by a fill kernel, an eager allocation-free call on other inputs that
    reuses the scratch array, an eager ozfp4_dgemm) and synchronizations:
    every replay gives the eager result bit for bit."""
    import torch
    assert gpu_lib.ozfp4_init() == gpu_lib.OZFP4_OK
    m, n, k, L = 300, 260, 500, 18
    A, B = dgemm_inputs(m, n, k, 0.5, SEED + 5)
    Ad, Bd = dev_cm(A), dev_cm(B)
    want = o.dgemm(A, B, L)["C"]
    A2, B2 = dgemm_inputs(200, 100, 300, 0.5, SEED + 6)
    A2d, B2d = dev_cm(A2), dev_cm(B2)
    want2 = o.dgemm(A2, B2, 14)["C"]
    C = torch.zeros((n, m), dtype=torch.float64, device="cuda").t()
    C2 = torch.zeros((100, 200), dtype=torch.float64, device="cuda").t()
    # eager warm-up on a side stream before the capture
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        gpu_lib.ozfp4_set_stream(side.cuda_stream)
        assert _call_noalloc(gpu_lib, Ad, Bd, C, L) == gpu_lib.OZFP4_OK
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert bits_equal(to_np(C), want)
    graph = torch.cuda.CUDAGraph()
    announce("dgemm_noalloc under stream capture")
    with torch.cuda.graph(graph):
        gpu_lib.ozfp4_set_stream(torch.cuda.current_stream().cuda_stream)
        rc = _call_noalloc(gpu_lib, Ad, Bd, C, L)
    assert rc == gpu_lib.OZFP4_OK
    for r in range(3):
        C.fill_(float("nan"))
        torch.cuda.synchronize()
        announce(f"graph replay {r}")
        graph.replay()
        torch.cuda.synchronize()
        assert bits_equal(to_np(C), want), f"replay {r}"
        gpu_lib.ozfp4_set_stream(torch.cuda.current_stream().cuda_stream)
        assert _call_noalloc(gpu_lib, A2d, B2d, C2, 14) == gpu_lib.OZFP4_OK
        torch.cuda.synchronize()
        assert bits_equal(to_np(C2), want2)
        assert bits_equal(to_np(gpu_lib.dgemm(A2d, B2d, 14)), want2)
        torch.cuda.synchronize()
    del graph
