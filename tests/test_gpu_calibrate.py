"""GPU checks of the reference-measurement kernels (ozfp4_calib_*), which
take part in no product but whose rates the benchmark reports: the plain
FP4 GEMM must compute C = A B exactly (else its rate R means nothing), the
LDS-DMA read must read every byte once, and the register-only MFMA loop
must run and return finite sums."""

import numpy as np
import pytest

import oracle as o
from gpu_util import announce, unpack_planes

pytestmark = pytest.mark.gpu

_E2M1 = np.array([o.e2m1_decode(c) for c in range(16)], dtype=np.float64)


@pytest.mark.parametrize("m,n,k", [(256, 256, 384), (512, 768, 1024), (1024, 256, 2048)])
def test_plain_fp4_gemm_exact(gpu_lib, m, n, k):
    import torch
    rng = np.random.default_rng([7, m, n, k])
    pa = rng.integers(0, 256, m * k // 2, dtype=np.uint8)
    pb = rng.integers(0, 256, n * k // 2, dtype=np.uint8)
    Av = _E2M1[unpack_planes(pa.reshape(1, -1), m, k)[0]]   # (m, k) values
    Bv = _E2M1[unpack_planes(pb.reshape(1, -1), n, k)[0]]   # (n, k) values
    want = Av @ Bv.T                                          # exact: quarter units below 2^53
    announce(f"calib_gemm_fp4 m={m} n={n} k={k}")
    C = gpu_lib.calib_gemm_fp4(torch.from_numpy(pa).cuda(), torch.from_numpy(pb).cuda(), m, n, k)
    got = C.cpu().numpy().astype(np.float64)
    assert np.array_equal(got, want)


def test_dma_read_reads_every_byte_once(gpu_lib):
    import torch
    nbytes = (1 << 20) * 3 + 5 * 1024
    rng = np.random.default_rng(11)
    src = rng.integers(0, 256, nbytes, dtype=np.uint8)
    announce(f"calib_dma_read {nbytes} bytes")
    for blocks in (1, 7, 256):
        sink = gpu_lib.calib_dma_read(torch.from_numpy(src).cuda(), blocks).cpu().numpy()
        got = np.bitwise_xor.reduce(sink.view(np.uint32))
        assert got == np.bitwise_xor.reduce(src.view(np.uint32)), blocks


def test_mfma_loop_runs(gpu_lib):
    import torch
    announce("calib_mfma 256 blocks x 16 iterations")
    sink, flops = gpu_lib.calib_mfma(256, 16, seed=3)
    torch.cuda.synchronize()
    s = sink.cpu().numpy()
    assert flops == 256 * 8 * 16 * 32 * 131072
    assert np.all(np.isfinite(s)) and np.count_nonzero(s) > s.size // 2


def test_mfma_loop_on_codes_exact(gpu_lib):
    """With every code E2M1 1.0 (nibble 2) each MFMA adds 64 to each of its
    outputs, and the rotations keep the codes, so every thread's checksum is
    (2 + 4 + 2) x 4 tiles x 16 values x 64 x iterations = 32768 iterations
    (exact in FP32). With random codes the loop runs and returns finite
    sums."""
    import torch
    iters = 16
    ones = torch.full((64,), 0x22222222, dtype=torch.int32, device="cuda")
    announce("calib_mfma_codes on code 1.0")
    sink, flops = gpu_lib.calib_mfma_codes(8, iters, ones, ones.clone())
    torch.cuda.synchronize()
    assert flops == 8 * 8 * iters * 32 * 131072
    assert np.all(sink.cpu().numpy() == 32768.0 * iters)
    g = torch.Generator(device="cpu").manual_seed(5)
    ca = torch.randint(-2 ** 31, 2 ** 31, (4096,), dtype=torch.int64, generator=g).to(torch.int32).cuda()
    cb = torch.randint(-2 ** 31, 2 ** 31, (4096,), dtype=torch.int64, generator=g).to(torch.int32).cuda()
    announce("calib_mfma_codes on random codes")
    sink, _ = gpu_lib.calib_mfma_codes(256, iters, ca, cb)
    torch.cuda.synchronize()
    s = sink.cpu().numpy()
    assert np.all(np.isfinite(s)) and np.count_nonzero(s) > s.size // 2

