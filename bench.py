"""Benchmark of the Ozaki-II-on-FP4 FP64 matrix product on one MI355X.

A step is one ozfp4_dgemm call on the m = n = k = 16384 workload (entries
(U(0,1) - 0.5) exp(0.5 N(0,1)), fixed seed, inputs resident in HBM): line
maxima and shifts, fused conversion + residues + limb encoding of A and of
B, the fused residue GEMM over all moduli, and the exact CRT
reconstruction. The printed JSON line carries the emulated-DGEMM rate
2 m n k / t and the residue GEMM against the FP4 matrix-core peak (stage
time measured with HIP events on the library's stream over the timed
steps), next to two measured reference rates for the same chip and run:
the register-only FP4 MFMA loop with the GEMM's register tile (the rate
without any memory traffic) and a plain single-product FP4 GEMM through
the same LDS-DMA ring (the effective rate R of the runtime model,
Sec. VII-C). It also carries the runtime model as a prediction from the
measured R and copy bandwidth, the CPU oracle timed on a bounded sample
with one worker per core, a per-stage breakdown, native FP64 matrix
products timed with the same protocol, alternating with the emulation at
18 and 19 moduli, the accuracy at 17 and 18 moduli at 4096^3 (both
metrics: error normalized by sum |A||B|, and relative to the correctly
rounded product), Ozaki scheme I on the same limbs (checked bit for bit
against scheme II), the FP32 emulation beside native FP32 and the
INT8-on-FP4 path as context.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--moduli L]
                       [--size N] [--sweep] [--quick] [--copy-calibration]
                       [--no-cpu-baseline] [--no-native] [--no-karatsuba]
                       [--no-phi4] [--no-ozi] [--no-sgemm] [--no-table1]
                       [--no-paper-accuracy] [--no-reference-rates] [--no-sweep4096]
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

FP4_PEAK_TFLOPS = 10100.0       # MI355X dense FP4 matrix peak (published)
FP64_PEAK_TFLOPS = 78.6         # MI355X FP64 matrix peak (published)
HBM_PEAK_GBS = 8000.0
METRIC = "emulated DGEMM TFLOPS at N=16384 + % of FP4 MFMA peak, 1xMI355X"
CPU_SHARE = 16                  # host cores that go with one GPU

# HBM bytes per launch of the residue GEMM at m = n = k = 16384, 18 moduli,
# from rocprofv3 FETCH_SIZE / WRITE_SIZE runs (KiB per dispatch, raw), with
# the factors that turn each counter into bytes: what the same counter reads
# for kernels of known traffic in the same runs (a plain 1 GiB device copy
# for WRITE_SIZE; a 1 GiB read through the GEMM's own LDS-DMA path for
# FETCH_SIZE). Valid only for the GEMM source they were taken on, identified
# by the hash of its code. None: not yet taken on the current source.
MEASURED_TRAFFIC = {
    "kernel_source_sha256_16": "2196fa9c2efb6bb7",
    "workload": (16384, 16384, 16384, 18),
    # means over the four dispatches of one run
    "fetch_kib": 75_497_684, "write_kib": 4_738_460,
    # 1 GiB read through the LDS-DMA path: 524,304 KiB; plain 1 GiB copy:
    # 524,300 KiB read, 1,048,576 KiB written
    "fetch_factor": 2.0, "write_factor": 1.0,
    "profile": "profiles/k_gemm_res_dgemm_16384_L18.md",
}
SEED = 20260806

# The paper's own configuration (19 moduli) as its Table I prints it for
# OzII-FP4 on an RTX PRO 6000 Blackwell: (compute stage, total) equivalent
# TFLOP/s per N. Context for the same configuration here, not a target.
PAPER_TABLE1_TFLOPS = {4096: (16.28, 10.81), 8192: (17.11, 13.52), 16384: (17.31, 15.26)}


GEMM_SOURCES = (  # (file, first line of the section, first line after it)
    ("device_common.hpp", "// ------------------------------------------------------------ Sec. VI-D", None),
    ("kernels.hpp", "// The residue GEMM over all moduli", "// INT8 variant (Sec. III)"),
)


def code_only(text: str) -> str:
    """C++ source without its comments, white space collapsed: what the
    compiler sees, so that editing a comment keeps the hash."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash() -> str:
    """sha256 (16 hex digits) of the code of the residue GEMM (comments and
    white space ignored): the tile mapping, the MFMA and LDS-DMA helpers and
    the block tiles (device_common.hpp), and the kernel itself (kernels.hpp)."""
    import hashlib
    h = hashlib.sha256()
    for name, start, end in GEMM_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_06812_amd", "csrc", name), encoding="utf-8") as f:
            text = f.read()
        a = text.index(start)
        h.update(code_only(text[a:text.index(end) if end else len(text)]).encode())
    return h.hexdigest()[:16]


def measured_traffic(N, L):
    """The residue GEMM's HBM bytes per launch from the committed counters,
    or None if they were not taken on this source and workload."""
    t = MEASURED_TRAFFIC
    if t["kernel_source_sha256_16"] is None or kernel_source_hash() != t["kernel_source_sha256_16"] \
            or (N, N, N, L) != t["workload"]:
        return None
    read = t["fetch_kib"] * 1024.0 * t["fetch_factor"]
    write = t["write_kib"] * 1024.0 * t["write_factor"]
    return {"GB": (read + write) / 1e9, "read_GB": read / 1e9, "write_GB": write / 1e9,
            "fetch_size_kib_raw": t["fetch_kib"], "write_size_kib_raw": t["write_kib"],
            "fetch_factor": t["fetch_factor"], "write_factor": t["write_factor"],
            "source": t["profile"]}


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def dev_cm(X, torch):
    import numpy as np
    return torch.from_numpy(np.ascontiguousarray(X.T)).to("cuda").t()


def time_dgemm(ozfp4, torch, Ad, Bd, C, L, steps, warmup, profile=True):
    """The protocol of the contract: W untimed calls, then K calls bracketed
    by synchronisations. Returns (ms per step, mean stage ms)."""
    return time_call(ozfp4, torch, lambda: ozfp4.dgemm(Ad, Bd, L, out=C), steps, warmup, profile)


def time_call(ozfp4, torch, call, steps, warmup, profile=True):
    """time_dgemm for any library call (stage times from ozfp4_stage_times)."""
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    ozfp4.ozfp4_profile(profile)
    stage_sum = None
    t0 = time.perf_counter()
    for _ in range(steps):
        call()
        if profile:
            st = ozfp4.ozfp4_stage_times()
            stage_sum = st if stage_sum is None else [a + b for a, b in zip(stage_sum, st)]
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ozfp4.ozfp4_profile(False)
    stages = [s / steps for s in stage_sum] if stage_sum else None
    return (t1 - t0) * 1e3 / steps, stages


def event_ms(torch, fn):
    """GPU time of fn() on the current stream (HIP events), synchronized."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1)


def stats(xs):
    ys = sorted(xs)
    n = len(ys)
    med = ys[n // 2] if n % 2 else 0.5 * (ys[n // 2 - 1] + ys[n // 2])
    return {"median": med, "min": ys[0], "max": ys[-1], "mean": sum(ys) / n, "n": n}


def paired_times(torch, calls, rounds, warmup):
    """Times every call of `calls` (name -> function) `rounds` times with
    the same protocol: each call alone, bracketed by synchronisations, GPU
    time from HIP events on the current stream. The calls alternate, and
    the order rotates every round so no call always follows the same one.
    Returns name -> list of ms."""
    names = list(calls)
    for name in names:
        for _ in range(warmup):
            calls[name]()
    torch.cuda.synchronize()
    out = {n: [] for n in names}
    for r in range(rounds):
        k = r % len(names)
        for name in names[k:] + names[:k]:
            out[name].append(event_ms(torch, calls[name]))
    return out


def cpu_workers():
    """One worker per core of this process's CPU share."""
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        avail = os.cpu_count() or 1
    return max(1, min(avail, CPU_SHARE))


_POOL_AB = {}


def _oracle_tile(task):
    """Worker: the oracle on output rows r0:r1 and columns c0:c1 of the
    matrices inherited from the parent (whole rows of A and columns of B,
    so shifts and residues are those of the full problem)."""
    r0, r1, c0, c1, L = task
    import oracle
    from threadpoolctl import threadpool_limits
    A, B = _POOL_AB["A"], _POOL_AB["B"]
    with threadpool_limits(1):
        oracle.dgemm(A[r0:r1, :], B[:, c0:c1], L)
    return (r1 - r0) * (c1 - c0)


def cpu_baseline(A, B, L, k, budget_s=20.0, workers=None, max_side=4096):
    """The oracle, as it stands, on a bounded sample of output elements of
    the same workload: a square block of outputs at full k, split into
    tiles of at most 256 x 256 that a pool of `workers` processes (one per
    core, one BLAS thread each) computes in parallel; the block grows until
    one timed run takes at least half of `budget_s` seconds or reaches
    max_side. Run it before the process touches the GPU: the workers are
    forked and inherit A and B."""
    import multiprocessing as mp

    import numpy as np
    workers = workers or cpu_workers()
    _POOL_AB["A"], _POOL_AB["B"] = np.asarray(A), np.asarray(B)
    ctx = mp.get_context("fork")
    side, elapsed, first = 64, 0.0, None
    try:
        with ctx.Pool(workers) as pool:
            pool.map(_oracle_tile, [(0, 2, 0, 2, L)] * workers)   # workers up
            while True:
                t = min(256, side)
                tasks = [(r, r + t, c, c + t, L) for r in range(0, side, t) for c in range(0, side, t)]
                t0 = time.perf_counter()
                done = sum(pool.map(_oracle_tile, tasks, chunksize=1))
                elapsed = time.perf_counter() - t0
                assert done == side * side
                first = (side, elapsed) if first is None else first
                if elapsed >= budget_s / 2 or side >= max_side:
                    break
                side = min(max_side, side * (2 if elapsed > budget_s / 8 else 4))
    finally:
        _POOL_AB.clear()
    tflops = 2.0 * k * side * side / elapsed / 1e12
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        affinity = None
    return {"value": tflops, "unit": "TFLOP/s (emulated DGEMM)", "cores": workers,
            "kind": "oracle", "os_cpu_count": os.cpu_count(), "affinity_cpus": affinity,
            "sample": f"{side}x{side} output block of the {A.shape[0]}x{B.shape[1]}x{k} workload at full k, "
                      f"{L} moduli, {elapsed:.2f} s on {workers} worker processes (one per core of the "
                      f"CPU share, one BLAS thread each; tiles of up to 256x256 outputs; first size "
                      f"{first[0]}x{first[0]}: {first[1]:.2f} s)"}


def _line_integers(X):
    """Each line of X (the last axis runs along k) as integers times a power
    of two shared by the line: X = sign * N * 2^base, with N = M 2^sh, M the
    53-bit significand and sh >= 0 its offset above the line's lowest
    exponent. Returns (sign, M, sh, base)."""
    import numpy as np
    f, e = np.frexp(np.abs(X))
    M = np.ldexp(f, 53).astype(np.int64)
    E = e.astype(np.int64) - 53
    big = np.iinfo(np.int64).max
    Em = np.where(M == 0, big, E)
    base = Em.min(axis=-1, keepdims=True)
    base = np.where(base == big, 0, base)
    sh = np.where(M == 0, 0, E - base)
    return np.where(X < 0, -1, 1).astype(np.int64), M, sh, base[..., 0]


def _digit(M, sh, q, bits=18):
    """Digit q (bits [bits q, bits (q + 1))) of N = M 2^sh."""
    import numpy as np
    lo = bits * q - sh                       # where the digit starts within M
    Mu = M.astype(np.uint64)
    mask = np.uint64((1 << bits) - 1)
    down = (Mu >> np.clip(lo, 0, 63).astype(np.uint64)) & mask
    up = (Mu << np.clip(-lo, 0, 63).astype(np.uint64)) & mask
    return np.where(lo >= 53, 0, np.where(lo >= 0, down, np.where(lo <= -bits, 0, up))).astype(np.int64)


def exact_reference(A, B, rows, cols):
    """Exact (AB)_ij and sum_k |A_ik||B_kj| on the block rows x cols, as
    arrays of Fractions: every row of A and column of B becomes integers
    times a power of two, the integers are cut into 18-bit digits, and each
    pair of digit matrices is multiplied in FP64, exactly (every sum is
    below 2^36 k <= 2^53 for k < 2^17); the digit products are recombined
    with Python integers."""
    import numpy as np
    from fractions import Fraction
    Ab = np.asarray(A, dtype=np.float64)[np.asarray(rows), :]
    Bb = np.asarray(B, dtype=np.float64)[:, np.asarray(cols)].T.copy()   # lines along k
    k = Ab.shape[1]
    if k >= 1 << 17:
        raise ValueError("k too large for exact FP64 digit products")
    sa, Ma, sha, ba = _line_integers(Ab)
    sb, Mb, shb, bb = _line_integers(Bb)
    da = [_digit(Ma, sha, q) for q in range((53 + int(sha.max(initial=0)) + 17) // 18)]
    db = [_digit(Mb, shb, q) for q in range((53 + int(shb.max(initial=0)) + 17) // 18)]
    prod = np.zeros((Ab.shape[0], Bb.shape[0]), dtype=object)
    absum = np.zeros_like(prod)
    for p, x in enumerate(da):
        for q, y in enumerate(db):
            w = 1 << (18 * (p + q))
            sp = np.rint((sa * x).astype(np.float64) @ (sb * y).astype(np.float64).T)
            ap = np.rint(x.astype(np.float64) @ y.astype(np.float64).T)
            prod = prod + sp.astype(np.int64).astype(object) * w
            absum = absum + ap.astype(np.int64).astype(object) * w
    ex = np.empty(prod.shape, dtype=object)
    ab = np.empty(prod.shape, dtype=object)
    for i in range(prod.shape[0]):
        for j in range(prod.shape[1]):
            sc = Fraction(2) ** (int(ba[i]) + int(bb[j]))
            ex[i, j] = Fraction(int(prod[i, j])) * sc
            ab[i, j] = Fraction(int(absum[i, j])) * sc
    return ex, ab


def accuracy_bits(C_block, ref):
    """Maximum over the block of |C - AB| / sum |A||B| (Sec. VII-A), as
    -log2, and the maximum itself."""
    from fractions import Fraction
    exact, denom = ref
    worst = 0.0
    for i in range(exact.shape[0]):
        for j in range(exact.shape[1]):
            if denom[i, j] != 0:
                e = float(abs(Fraction(float(C_block[i, j])) - exact[i, j]) / denom[i, j])
                worst = max(worst, e)
    return (-math.log2(worst) if worst > 0 else float("inf")), worst


def elementwise_vs_rounded(C_block, ref):
    """Against fl(AB), the exact product rounded once to FP64: the maximum
    elementwise |C - fl(AB)| / |fl(AB)|, the fraction of elements within
    2^-50 of it, the fraction equal to it and the largest distance in units
    in the last place (elements with fl(AB) = 0 count as within 2^-50 and
    equal only if C is 0)."""
    import struct
    exact, _ = ref
    n = within = equal = 0
    worst, worst_ulps = 0.0, 0

    def key(x):   # monotone integer image of a double
        b = struct.unpack("<q", struct.pack("<d", x))[0]
        return b if b >= 0 else -(b & 0x7fffffffffffffff)
    for i in range(exact.shape[0]):
        for j in range(exact.shape[1]):
            fl = float(exact[i, j])
            c = float(C_block[i, j])
            n += 1
            if fl == 0.0:
                within += c == 0.0
                equal += c == 0.0
                continue
            rel = abs(c - fl) / abs(fl)
            worst = max(worst, rel)
            within += rel <= 2.0 ** -50
            equal += c == fl
            worst_ulps = max(worst_ulps, abs(key(c) - key(fl)))
    return {"metric": "max_ij |C_ij - fl(AB)_ij| / |fl(AB)_ij|, fl = exact product rounded once",
            "max_rel_error": worst, "error_bits": -math.log2(worst) if worst > 0 else float("inf"),
            "frac_within_2^-50": within / n, "frac_equal_to_fl": equal / n, "max_ulps": worst_ulps}


def block_of(C, rows, cols, torch):
    r = torch.as_tensor(rows, device="cuda")
    c = torch.as_tensor(cols, device="cuda")
    return C[r][:, c].cpu().numpy()


def measure_attainable(ozfp4, torch, target_ms=80.0, reps=3):
    """The register-only FP4 MFMA loop (one block of eight waves per CU, the
    residue GEMM's register tile and product order, operands changed every
    k fragment) sustained over about target_ms per launch: the matrix-core
    rate this chip holds with no memory traffic."""
    blocks = 256
    iters = 256
    ozfp4.calib_mfma(blocks, iters)
    t = event_ms(torch, lambda: ozfp4.calib_mfma(blocks, iters))
    iters = max(1, int(iters * target_ms / max(t, 1e-3)))
    flops = blocks * 8 * iters * 32 * 131072.0
    times = [event_ms(torch, lambda: ozfp4.calib_mfma(blocks, iters)) for _ in range(reps)]
    st = stats(times)
    return {"tflops": flops / st["median"] / 1e9, "frac": flops / st["median"] / 1e9 / FP4_PEAK_TFLOPS,
            "ms": st, "flops_per_launch": flops, "blocks": blocks, "iterations": iters,
            "kernel": "k_calib_mfma (ozfp4_calib_mfma)"}


def limb_codes(ozfp4, torch, Ad, Bd, L, lines=256):
    """The workload's own E2M1 codes for the code-driven MFMA loop: the limb
    planes of the first `lines` rows of A and columns of B at full k (their
    shifts are the whole matrices', since a row or column is whole), c0 and
    c1 planes of every modulus, interleaved as 8 words of c0 and 8 of c1 per
    lane (the order a[p][i][w] of ozfp4_calib_mfma_codes)."""
    pa, pb = ozfp4.limb_planes(Ad[:lines, :], Bd[:, :lines], L)

    def interleave(planes):
        w = planes.view(torch.int32)   # (planes, words)
        c0 = w[0::2].reshape(-1, 8)
        c1 = w[1::2].reshape(-1, 8)
        n = min(c0.shape[0], c1.shape[0])
        return torch.cat([c0[:n], c1[:n]], dim=1).reshape(-1).contiguous()
    return interleave(pa), interleave(pb)


def measure_attainable_codes(ozfp4, torch, codes_a, codes_b, target_ms=80.0, reps=3):
    """The register-only loop of measure_attainable on the workload's own
    limb codes (rotated by whole codes every k fragment), since the power the
    matrix cores draw, and so the clock they hold, depends on the data."""
    blocks = 256
    iters = 256
    ozfp4.calib_mfma_codes(blocks, iters, codes_a, codes_b)
    t = event_ms(torch, lambda: ozfp4.calib_mfma_codes(blocks, iters, codes_a, codes_b))
    iters = max(1, int(iters * target_ms / max(t, 1e-3)))
    flops = blocks * 8 * iters * 32 * 131072.0
    times = [event_ms(torch, lambda: ozfp4.calib_mfma_codes(blocks, iters, codes_a, codes_b))
             for _ in range(reps)]
    st = stats(times)
    return {"tflops": flops / st["median"] / 1e9, "frac": flops / st["median"] / 1e9 / FP4_PEAK_TFLOPS,
            "ms": st, "flops_per_launch": flops, "blocks": blocks, "iterations": iters,
            "codes": "limb planes of the first 256 rows of A and columns of B, every modulus",
            "kernel": "k_calib_mfma_codes (ozfp4_calib_mfma_codes)"}


def measure_plain_gemm(ozfp4, torch, N=16384, target_ms=100.0):
    """R of the runtime model: a plain single-product FP4 GEMM (C = A B in
    FP32 from one plane of random E2M1 codes each) at N^3, streamed through
    the same LDS-DMA ring as the residue GEMM, launched back to back for
    about target_ms; rate = 2 N^3 per launch over the mean launch time."""
    import numpy as np
    rng = np.random.default_rng(SEED + 90)
    pa = torch.from_numpy(rng.integers(0, 256, N * N // 2, dtype=np.uint8)).cuda()
    pb = torch.from_numpy(rng.integers(0, 256, N * N // 2, dtype=np.uint8)).cuda()
    C = torch.empty_strided((N, N), (1, N), dtype=torch.float32, device="cuda")
    for _ in range(2):
        ozfp4.calib_gemm_fp4(pa, pb, N, N, N, out=C)
    t1 = event_ms(torch, lambda: ozfp4.calib_gemm_fp4(pa, pb, N, N, N, out=C))
    reps = max(3, int(math.ceil(target_ms / max(t1, 1e-3))))

    def run():
        for _ in range(reps):
            ozfp4.calib_gemm_fp4(pa, pb, N, N, N, out=C)
    t = event_ms(torch, run)
    del pa, pb, C
    ms = t / reps
    return {"tflops": 2.0 * N ** 3 / ms / 1e9, "frac": 2.0 * N ** 3 / ms / 1e9 / FP4_PEAK_TFLOPS,
            "ms_per_launch": ms, "launches": reps, "workload": f"fp4 gemm {N}^3, fp32 out",
            "kernel": "k_calib_gemm_fp4 (ozfp4_calib_gemm_fp4)"}


def measure_copy_beta(torch, reps=21):
    """beta of the runtime model: a plain 1 GiB device copy, read plus
    written bytes over its time (the paper's copy benchmark), the median
    of `reps` copies each timed alone with HIP events."""
    src = torch.empty(1 << 27, dtype=torch.float64, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    ms = stats([event_ms(torch, lambda: dst.copy_(src)) for _ in range(reps)])["median"]
    beta = 2.0 * src.numel() * 8 / (ms * 1e-3) / 1e9
    del src, dst
    return beta


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=12)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--moduli", type=int, default=18)
    ap.add_argument("--size", type=int, default=16384)
    ap.add_argument("--sweep", action="store_true", help="sweep 12..20 moduli at the given size")
    ap.add_argument("--quick", action="store_true",
                    help="the headline, the reference rates and the model only (profiling runs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-native", action="store_true")
    ap.add_argument("--no-int8", action="store_true")
    ap.add_argument("--no-accuracy", action="store_true")
    ap.add_argument("--no-reference-rates", action="store_true",
                    help="skip the register-only MFMA loop, the plain FP4 GEMM and the copy bandwidth")
    ap.add_argument("--no-sweep4096", action="store_true",
                    help="skip the 17 / 18 moduli accuracy check at 4096^3")
    ap.add_argument("--no-phi4", action="store_true",
                    help="skip the phi = 4 workload (8192 x 8192 x 32768) at both capacity caps")
    ap.add_argument("--no-karatsuba", action="store_true",
                    help="skip timing the three-product Karatsuba mode (comparison only)")
    ap.add_argument("--no-ozi", action="store_true",
                    help="skip Ozaki scheme I (15 limbs) and its bitwise check against scheme II")
    ap.add_argument("--no-sgemm", action="store_true",
                    help="skip the FP32 emulation (ozfp4_sgemm) and native FP32 on FP32 copies of the inputs")
    ap.add_argument("--no-paper-accuracy", action="store_true",
                    help="skip the paper's accuracy experiment (its input law, K = 8192, 128 x 128)")
    ap.add_argument("--no-table1", action="store_true",
                    help="skip the paper's configuration (19 moduli) at N = 4096, 8192, 16384")
    ap.add_argument("--no-one-limb", action="store_true",
                    help="skip the one-limb moduli list (11 first, one FP4 product for it)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy and a 1 GiB read through the LDS-DMA path "
                         "(known traffic for the HBM byte counters)")
    args = ap.parse_args()
    if args.quick:
        for name in ("cpu_baseline", "native", "int8", "accuracy", "sweep4096", "phi4", "karatsuba",
                     "ozi", "sgemm", "paper_accuracy", "table1", "one_limb"):
            setattr(args, "no_" + name, True)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this method has no multi-GPU path "
              "(its output tiles and moduli would shard without communication)",
              file=sys.stderr)
        return 2

    import numpy as np

    from paper_2608_06812_amd.workloads import dgemm_inputs, int8_inputs, paper_law_inputs
    N = args.size
    L = args.moduli

    log(f"generating inputs {N}^3")
    A, B = dgemm_inputs(N, N, N, 0.5, SEED + 2)

    cpu_rec = None
    if not args.no_cpu_baseline and not args.sweep:
        # before the process touches the GPU: the pool's workers are forked
        log(f"timing the CPU oracle on a sample ({cpu_workers()} workers)")
        cpu_rec = cpu_baseline(A, B, L, N)
        log(json.dumps(cpu_rec))

    import torch

    from paper_2608_06812_amd import ozfp4
    ozfp4.load()
    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    torch.cuda.set_device(0)

    Ad, Bd = dev_cm(A, torch), dev_cm(B, torch)
    C = torch.empty_strided((N, N), (1, N), dtype=torch.float64, device="cuda")

    def with_heads(h, call):
        """call() with the moduli list of h one-limb heads (11, 9, 8, 7, 5
        first), then the greedy list again."""
        ozfp4.ozfp4_set_one_limb_moduli(h)
        try:
            return call()
        finally:
            ozfp4.ozfp4_set_one_limb_moduli(0)

    def one_limb(call):
        return with_heads(1, call)

    # one-limb lists reported beside the headline: (heads, moduli, the greedy
    # list whose capacities, and hence C, they reproduce at 16384^3)
    HEAD_LISTS = [(1, 18, None), (5, 21, 18), (4, 21, 19)]

    if args.sweep:
        # accuracy on a 128 x 128 output block at full k (all 16384 elements)
        rows = np.arange(128)
        cols = np.arange(128)
        log("exact reference block")
        ref = exact_reference(A, B, rows, cols)
        out = []
        for Ls in range(12, 21):
            try:
                ms, st = time_dgemm(ozfp4, torch, Ad, Bd, C, Ls, max(2, args.steps // 3), 1)
            except ozfp4.OzFP4Error as err:
                log(f"{Ls} moduli: {err}")
                continue
            Cb = block_of(C, rows, cols, torch)
            bits, worst = accuracy_bits(Cb, ref)
            rec = {"n_moduli": Ls, "ms": ms, "tflops": 2.0 * N ** 3 / ms / 1e9,
                   "gemm_ms": st[3], "error_bits": bits, "max_normalized_error": worst,
                   "fp64_accurate": worst <= 2.0 ** -50,
                   "vs_rounded_product": elementwise_vs_rounded(Cb, ref)}
            log(json.dumps(rec))
            out.append(rec)
        accurate = [r["n_moduli"] for r in out if r["fp64_accurate"]]
        print(json.dumps({"sweep": out, "size": N, "block": "128x128",
                          "smallest_fp64_accurate_moduli": min(accurate) if accurate else None}))
        return 0

    log(f"timing ozfp4_dgemm, {L} moduli")
    ms, stages = time_dgemm(ozfp4, torch, Ad, Bd, C, L, args.steps, args.warmup)
    value = 2.0 * N ** 3 / ms / 1e9
    gemm_ms = stages[3]
    # three limb products per modulus plus a1 b1 for every modulus but 169,
    # where 169 a1 b1 vanishes mod 169 and is not executed
    Q = 4 * L - 1
    flops_exec = Q * 2.0 * N ** 3
    achieved = flops_exec / gemm_ms / 1e9
    stage_names = ["scale", "encode_A", "encode_B", "residue_gemm", "crt"]
    log(f"{ms:.2f} ms per call, residue GEMM {gemm_ms:.2f} ms ({achieved:.0f} TFLOP/s)")

    # memory-bound stages: algorithmic bytes per call
    bytes_scale = 8.0 * (N * N + N * N)
    bytes_enc = 8.0 * N * N + 2 * L * N * N / 2.0   # per operand: read FP64, write 2L planes
    bytes_crt = L * N * N + 8.0 * N * N
    hbm = {
        "scale_GBs": bytes_scale / stages[0] / 1e6,
        "encode_A_GBs": bytes_enc / stages[1] / 1e6,
        "encode_B_GBs": bytes_enc / stages[2] / 1e6,
        "crt_GBs": bytes_crt / stages[4] / 1e6,
    }
    # bytes of the memory-bound work of one call: scale, both encodes, the
    # residues the GEMM writes, the CRT
    D = bytes_scale + 2 * bytes_enc + L * N * N + bytes_crt
    traffic = measured_traffic(N, L)

    result = {
        "metric": METRIC, "value": value, "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64",
        "arithmetic": "FP4 E2M1 MFMA products, FP32 accumulation, exact integer CRT",
        "data": "synthetic: (U(0,1)-0.5)*exp(0.5*N(0,1)), seed %d" % (SEED + 2),
        "config": {"workload": f"dgemm m=n=k={N}, phi=0.5", "m": N, "n": N, "k": N,
                   "n_moduli": L, "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "kernel": "k_gemm_res", "achieved": achieved,
                     "peak": FP4_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": achieved / FP4_PEAK_TFLOPS,
                     "traffic": traffic["GB"] if traffic else None,
                     "traffic_unit": "GB per launch (HBM read + write)",
                     "traffic_detail": traffic,
                     "algorithmic_GB": (2 * L * N * N + L * N * N) / 1e9,
                     "flops_per_launch": flops_exec, "products_per_element": Q,
                     "avg_launch_ms": gemm_ms},
        "stages_ms": dict(zip(stage_names, stages)),
        "hbm_GBs": hbm,
        "compute_stage_tflops": 2.0 * N ** 3 / (gemm_ms + stages[4]) / 1e9,
    }

    # the paper's runtime model t = 2 Q N^3 / R + D / beta (Eq. (model)):
    # at the published peaks, and as a prediction from rates measured here
    # on other kernels (R: the plain FP4 GEMM; beta: a device copy)
    result["model"] = {"Q": Q, "D_GB": D / 1e9,
                       "ms_at_published_peaks": (flops_exec / (FP4_PEAK_TFLOPS * 1e12) +
                                                 D / (HBM_PEAK_GBS * 1e9)) * 1e3}
    if not args.no_reference_rates:
        log("reference rates: register-only MFMA loop, plain FP4 GEMM, device copy")
        att = measure_attainable(ozfp4, torch)
        codes_a, codes_b = limb_codes(ozfp4, torch, Ad, Bd, L)
        att_codes = measure_attainable_codes(ozfp4, torch, codes_a, codes_b)
        del codes_a, codes_b
        plain = measure_plain_gemm(ozfp4, torch)
        beta = measure_copy_beta(torch)
        result["roofline"]["attainable"] = att["tflops"]
        result["roofline"]["attainable_frac"] = att["frac"]
        result["roofline"]["frac_of_attainable"] = achieved / att["tflops"]
        result["roofline"]["attainable_limb_codes"] = att_codes["tflops"]
        result["roofline"]["frac_of_attainable_limb_codes"] = achieved / att_codes["tflops"]
        result["roofline"]["plain_fp4_gemm"] = plain["tflops"]
        result["roofline"]["frac_of_plain_fp4_gemm"] = achieved / plain["tflops"]
        result["reference_rates"] = {"mfma_loop": att, "mfma_loop_limb_codes": att_codes,
                                     "plain_fp4_gemm": plain, "copy_GBs": beta}
        t_gemm = flops_exec / (plain["tflops"] * 1e12) * 1e3
        t_pre = D / (beta * 1e9) * 1e3
        result["hbm_copy_GBs"] = beta
        result["hbm_frac_of_copy"] = {k.replace("_GBs", ""): v / beta for k, v in hbm.items()}
        result["model"].update({
            "R_tflops": plain["tflops"], "beta_GBs": beta,
            "predicted_ms": t_gemm + t_pre, "predicted_gemm_ms": t_gemm, "predicted_pre_ms": t_pre,
            "measured_ms": ms, "measured_over_predicted": ms / (t_gemm + t_pre),
            "measured_gemm_over_predicted": gemm_ms / t_gemm})
        log(json.dumps({"attainable": att["tflops"], "attainable_limb_codes": att_codes["tflops"],
                        "R": plain["tflops"], "beta": beta,
                        "model": result["model"]}))

    if args.copy_calibration:
        # known traffic for the byte counters: a plain 1 GiB device copy (the
        # normal load and store path) and a 1 GiB read through the LDS-DMA
        # path of the residue GEMM
        src = torch.empty(1 << 27, dtype=torch.float64, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        src8 = src.view(torch.uint8)[: (1 << 30) - 1024]
        for _ in range(3):
            ozfp4.calib_dma_read(src8, 2048)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = {"copy_read": src.numel() * 8, "copy_write": dst.numel() * 8,
                                            "dma_read": src8.numel()}
        del src, dst, src8

    ref_block = None
    if not args.no_accuracy:
        rows = np.arange(0, N, N // 128)[:128]
        cols = np.arange(0, N, N // 128)[:128]
        ref_block = exact_reference(A, B, rows, cols)
        Cb = block_of(C, rows, cols, torch)
        bits, worst = accuracy_bits(Cb, ref_block)
        result["accuracy"] = {"block": "128x128 (every N/128-th row and column)",
                              "metric": "max_ij |C_ij - (AB)_ij| / sum_k |A_ik||B_kj| (Sec. VII-A)",
                              "error_bits": bits, "max_normalized_error": worst,
                              "fp64_accurate": worst <= 2.0 ** -50,
                              "vs_rounded_product": elementwise_vs_rounded(Cb, ref_block)}

    if not args.no_native:
        # native FP64 matmul and the emulation at 18 and 19 moduli, timed
        # with one protocol: each call alone between synchronisations, GPU
        # time from HIP events, the three alternating in one loop
        log("native FP64 torch.matmul alternating with the emulation at 18 and 19 moduli")
        Ar = torch.from_numpy(A).to("cuda")
        Br = torch.from_numpy(B).to("cuda")
        Cn = torch.empty((N, N), dtype=torch.float64, device="cuda")
        calls = {"emulation_L18": lambda: ozfp4.dgemm(Ad, Bd, 18, out=C),
                 "native_fp64": lambda: torch.matmul(Ar, Br, out=Cn),
                 "emulation_L19": lambda: ozfp4.dgemm(Ad, Bd, 19, out=C)}
        if not args.no_one_limb:
            for h_, L_, _ in HEAD_LISTS:
                calls[f"emulation_heads{h_}_L{L_}"] = (
                    lambda h_=h_, L_=L_: with_heads(h_, lambda: ozfp4.dgemm(Ad, Bd, L_, out=C)))
        rounds = max(5, args.steps)
        times = paired_times(torch, calls, rounds, max(2, args.warmup))
        st = {name: stats(v) for name, v in times.items()}
        nat = st["native_fp64"]
        cmp = {}
        for key in [n for n in calls if n != "native_fp64"]:
            em = st[key]
            ratio = nat["median"] / em["median"]
            cmp[key.replace("emulation_", "")] = {
                "speedup_of_emulation": ratio,
                "emulation_ms": em, "emulation_tflops": 2.0 * N ** 3 / em["median"] / 1e9,
                # a win only if every native call was slower than every emulated one
                "faster_beyond_spread": nat["min"] > em["max"],
                "reading": ("emulation faster than native FP64, beyond the spread of both"
                            if nat["min"] > em["max"] else
                            "slower than native FP64" if ratio < 1.0 else
                            "median faster, but within the spread of the two")}
        result["native_fp64"] = {"protocol": f"{rounds} rounds, each call alone between synchronisations, "
                                             f"HIP events, calls alternating (order rotated per round)",
                                 "ms": nat, "tflops": 2.0 * N ** 3 / nat["median"] / 1e9,
                                 "speedup_of_emulation": cmp["L18"]["speedup_of_emulation"],
                                 "vs_emulation": cmp}
        log(json.dumps(result["native_fp64"]))
        if ref_block is not None:
            # native FP64 accumulates rounding errors along k; same block
            torch.matmul(Ar, Br, out=Cn)
            Cnb = block_of(Cn, rows, cols, torch)
            nbits, nworst = accuracy_bits(Cnb, ref_block)
            result["native_fp64"].update({"error_bits": nbits, "max_normalized_error": nworst,
                                          "vs_rounded_product": elementwise_vs_rounded(Cnb, ref_block)})
        # leave the default output in C
        ozfp4.dgemm(Ad, Bd, L, out=C)
        del Ar, Br, Cn
        torch.cuda.empty_cache()

    if not args.no_one_limb:
        # the one-limb moduli lists: h one-limb heads (one FP4 product each)
        # and the two-limb moduli by the greedy rule seeded with them;
        # reported beside the headline. Where a list's capacities equal a
        # greedy list's, its C must equal that list's bit for bit.
        Cg = {L: C.clone()}
        lists = {}
        for h_, L_, same_as in HEAD_LISTS:
            if same_as is not None and same_as not in Cg:
                Cg[same_as] = torch.empty_like(C)
                ozfp4.dgemm(Ad, Bd, same_as, out=Cg[same_as])
            log(f"one-limb moduli list: {h_} heads, {L_} moduli")
            oms, ost = with_heads(h_, lambda: time_call(
                ozfp4, torch, lambda: ozfp4.dgemm(Ad, Bd, L_, out=C), args.steps, args.warmup))
            mods = with_heads(h_, lambda: ozfp4.ozfp4_moduli(L_))
            nh = min(h_, L_)
            # two-limb moduli: four products each, 169 three; heads: one
            q = sum(3 if x == 169 else 4 for x in mods[nh:]) + nh
            rec = {"heads": h_, "n_moduli": L_, "moduli": mods,
                   "capacity_bits": list(with_heads(h_, lambda: ozfp4.ozfp4_capacity(N, L_))),
                   "ms": oms, "tflops": 2.0 * N ** 3 / oms / 1e9,
                   "stages_ms": dict(zip(stage_names, ost)),
                   "limb_products_per_element": q, "headline_products_per_element": Q,
                   "gemm_fp4_tflops": q * 2.0 * N ** 3 / ost[3] / 1e9,
                   "speedup_vs_headline": ms / oms}
            if same_as is not None:
                rec["c_bitwise_equal_to_greedy"] = {
                    "n_moduli": same_as,
                    "equal": bool(torch.equal(C.view(torch.int64), Cg[same_as].view(torch.int64)))}
            if ref_block is not None:
                Cb1 = block_of(C, rows, cols, torch)
                b1, w1 = accuracy_bits(Cb1, ref_block)
                rec.update({"error_bits": b1, "max_normalized_error": w1,
                            "fp64_accurate": w1 <= 2.0 ** -50})
            if "native_fp64" in result:
                rec["vs_native_fp64"] = result["native_fp64"]["vs_emulation"].get(f"heads{h_}_L{L_}")
            lists[f"heads{h_}_L{L_}"] = rec
            log(json.dumps(rec))
        result["one_limb"] = lists
        # the headline's own output (bit for bit) by the faster list, if any
        same = [r for r in lists.values()
                if r.get("c_bitwise_equal_to_greedy", {}).get("n_moduli") == L
                and r["c_bitwise_equal_to_greedy"]["equal"]]
        if same:
            r = min(same, key=lambda x: x["ms"])
            nat_cmp = r.get("vs_native_fp64") or {}
            result["headline_output_by_one_limb_heads"] = {
                "heads": r["heads"], "n_moduli": r["n_moduli"], "ms": r["ms"], "tflops": r["tflops"],
                "c_bitwise_equal_to_headline": True, "speedup_vs_headline": r["speedup_vs_headline"],
                "vs_native_fp64": nat_cmp.get("speedup_of_emulation"),
                "faster_than_native_beyond_spread": nat_cmp.get("faster_beyond_spread")}
        C.copy_(Cg[L])
        del Cg
        torch.cuda.empty_cache()

    if not args.no_sweep4096:
        # the moduli count of the headline: the smallest count whose output
        # is FP64-accurate at 4096^3 (error normalized by sum |A||B| on an
        # exact 128 x 128 block at most 2^-50); 17 must fail, 18 pass
        log("accuracy at 4096^3 with 17 and 18 moduli")
        N2 = 4096
        A2, B2 = dgemm_inputs(N2, N2, N2, 0.5, SEED + 5)
        A2d, B2d = dev_cm(A2, torch), dev_cm(B2, torch)
        C2 = torch.empty_strided((N2, N2), (1, N2), dtype=torch.float64, device="cuda")
        rows2 = np.arange(128)
        ref2 = exact_reference(A2, B2, rows2, rows2)
        sw = []
        for L2 in (17, 18):
            ms2, st2 = time_dgemm(ozfp4, torch, A2d, B2d, C2, L2, 10, 2)
            Cb2 = block_of(C2, rows2, rows2, torch)
            bits2, worst2 = accuracy_bits(Cb2, ref2)
            sw.append({"n_moduli": L2, "capacity_bits": list(ozfp4.ozfp4_capacity(N2, L2)),
                       "ms": ms2, "tflops": 2.0 * N2 ** 3 / ms2 / 1e9,
                       "error_bits": bits2, "max_normalized_error": worst2,
                       "fp64_accurate": worst2 <= 2.0 ** -50,
                       "vs_rounded_product": elementwise_vs_rounded(Cb2, ref2)})
            log(json.dumps(sw[-1]))
        ok = [r["n_moduli"] for r in sw if r["fp64_accurate"]]
        result["sweep4096"] = {"workload": "dgemm m=n=k=4096, phi=0.5", "block": "128x128 (rows and "
                               "columns 0..127)", "runs": sw,
                               "smallest_fp64_accurate_moduli": min(ok) if ok else None,
                               "headline_moduli_is_smallest": (ok == [18])}
        if not args.no_one_limb:
            sw1 = []
            for h2, L2 in ((1, 17), (1, 18), (5, 20), (5, 21)):
                ms2, _ = with_heads(h2, lambda: time_dgemm(ozfp4, torch, A2d, B2d, C2, L2, 10, 2))
                Cb2 = block_of(C2, rows2, rows2, torch)
                bits2, worst2 = accuracy_bits(Cb2, ref2)
                sw1.append({"heads": h2, "n_moduli": L2,
                            "capacity_bits": list(with_heads(h2, lambda: ozfp4.ozfp4_capacity(N2, L2))),
                            "ms": ms2, "tflops": 2.0 * N2 ** 3 / ms2 / 1e9,
                            "error_bits": bits2, "max_normalized_error": worst2,
                            "fp64_accurate": worst2 <= 2.0 ** -50})
                log(json.dumps(sw1[-1]))
            result["sweep4096"]["one_limb_runs"] = sw1
        del A2d, B2d, C2
        torch.cuda.empty_cache()

    if not args.no_karatsuba:
        # the Karatsuba mode of Sec. V-A (three products for the sum-limb
        # moduli): reported beside the default route, not as the headline
        log("timing the Karatsuba mode")
        Cref = C.clone()
        ozfp4.ozfp4_set_karatsuba(True)
        try:
            nplanes, _ = ozfp4.ozfp4_plane_count(L)
            kms, kst = time_dgemm(ozfp4, torch, Ad, Bd, C, L, max(3, args.steps // 2), 1)
        finally:
            ozfp4.ozfp4_set_karatsuba(False)
        nk = nplanes - 2 * L
        kprod = 4 * L - 1 - nk
        result["karatsuba"] = {
            "ms": kms, "tflops": 2.0 * N ** 3 / kms / 1e9, "gemm_ms": kst[3],
            "products_per_element": kprod, "default_products_per_element": 4 * L - 1,
            "fp4_tflops_gemm": kprod * 2.0 * N ** 3 / kst[3] / 1e9,
            "c_bitwise_equal_to_default": bool(torch.equal(Cref.view(torch.int64),
                                                           C.view(torch.int64)))}
        del Cref

    if not args.no_ozi:
        # Ozaki scheme I on the same limbs (Sec. IV): 15 limbs, 225 limb
        # products; its C is compared bit for bit with scheme II at 19
        # moduli, where both convert with 53-bit capacities (Sec. VII-A)
        log("scheme II with 19 moduli, then timing ozfp4_dgemm_ozi with 15 limbs")
        C19 = torch.empty_strided((N, N), (1, N), dtype=torch.float64, device="cuda")
        ozfp4.dgemm(Ad, Bd, 19, out=C19)
        oms, ost = time_call(ozfp4, torch, lambda: ozfp4.dgemm_ozi(Ad, Bd, 15, out=C),
                             max(3, args.steps // 4), 1)
        flops_ozi = 225 * 2.0 * N ** 3
        result["ozi"] = {
            "workload": f"dgemm m=n=k={N}, phi=0.5, scheme I, 15 limbs", "ms": oms,
            "tflops": 2.0 * N ** 3 / oms / 1e9, "products_per_element": 225,
            "stages_ms": dict(zip(["scale", "encode_A", "encode_B", "limb_gemm", "reduce"], ost)),
            "fp4_tflops_gemm": flops_ozi / ost[3] / 1e9,
            "fp4_frac": flops_ozi / ost[3] / 1e9 / FP4_PEAK_TFLOPS,
            "c_bitwise_equal_to_scheme2_19_moduli": bool(torch.equal(C.view(torch.int64),
                                                                     C19.view(torch.int64)))}
        log(json.dumps(result["ozi"]))
        del C19
        torch.cuda.empty_cache()

    if not args.no_paper_accuracy:
        # the paper's accuracy experiment: entries +-(1 + u) 2^e, e uniform in
        # {0..phi}, K = 8192, a 128 x 128 output, 19 moduli; max normalized
        # error over all 16384 outputs against the exact product
        log("paper accuracy experiment (phi = 0, 4, 32)")
        pa_runs = []
        for phi in (0, 4, 32):
            Ap, Bp = paper_law_inputs(128, 128, 8192, phi, SEED + 50 + phi)
            Cp = ozfp4.dgemm(dev_cm(Ap, torch), dev_cm(Bp, torch), 19)
            allr = np.arange(128)
            pbits, pworst = accuracy_bits(Cp.cpu().numpy(), exact_reference(Ap, Bp, allr, allr))
            pa_runs.append({"phi": phi, "error_bits": pbits, "max_normalized_error": pworst})
        result["paper_accuracy"] = {
            "workload": "dgemm 128 x 128 x 8192, entries +-(1+u) 2^e, e in {0..phi}, 19 moduli",
            "paper": "Sec. VII-A: 58.2 bits at phi = 0, 52.3 bits at phi = 32",
            "runs": pa_runs}
        log(json.dumps(result["paper_accuracy"]))

    if not args.no_table1:
        # the paper's configuration at its three sizes: "compute" is the
        # residue GEMM plus the CRT (the paper's compute stage), "total" the
        # whole call
        log("paper configuration (19 moduli) at N = 4096, 8192, 16384")
        rows1 = []
        for N1 in sorted(PAPER_TABLE1_TFLOPS):
            if N1 == N:
                A1d, B1d, C1 = Ad, Bd, C
            else:
                A1, B1 = dgemm_inputs(N1, N1, N1, 0.5, SEED + 3)
                A1d, B1d = dev_cm(A1, torch), dev_cm(B1, torch)
                C1 = torch.empty_strided((N1, N1), (1, N1), dtype=torch.float64, device="cuda")
            reps = max(5, int(2000 // (N1 / 1024) ** 3))
            t1, st1 = time_call(ozfp4, torch, lambda: ozfp4.dgemm(A1d, B1d, 19, out=C1), reps, 2)
            f1 = 2.0 * N1 ** 3
            comp, total = PAPER_TABLE1_TFLOPS[N1]
            rows1.append({"n": N1, "ms": t1, "tflops_total": f1 / t1 / 1e9,
                          "tflops_compute": f1 / (st1[3] + st1[4]) / 1e9,
                          "paper_tflops_compute": comp, "paper_tflops_total": total})
            if not args.no_one_limb:
                # the same C from 21 moduli with the one-limb heads 11, 9, 8, 7
                # (their capacities equal the 19 greedy moduli's at these k)
                C19 = C1.clone()
                t4, st4 = with_heads(4, lambda: time_call(
                    ozfp4, torch, lambda: ozfp4.dgemm(A1d, B1d, 21, out=C1), reps, 2))
                rows1[-1]["four_heads_21_moduli"] = {
                    "ms": t4, "tflops_total": f1 / t4 / 1e9,
                    "tflops_compute": f1 / (st4[3] + st4[4]) / 1e9,
                    "c_bitwise_equal_to_19_moduli": bool(torch.equal(C1.view(torch.int64),
                                                                     C19.view(torch.int64)))}
                C1.copy_(C19)
                del C19
            log(json.dumps(rows1[-1]))
            if N1 != N:
                del A1d, B1d, C1
        result["table1"] = {"workload": "dgemm m=n=k=N, phi=0.5, 19 moduli (the paper's configuration)",
                            "paper": "Table I, OzII-FP4, RTX PRO 6000 Blackwell (other hardware)",
                            "runs": rows1}
        torch.cuda.empty_cache()

    if not args.no_sgemm:
        # FP32 emulation on FP32 copies of the same inputs, with the fewest
        # moduli that give 24-bit capacities, beside native FP32 matmul
        L32 = ozfp4.sgemm_moduli(N)
        log(f"timing ozfp4_sgemm, {L32} moduli, and native FP32 torch.matmul")
        A32 = A.astype(np.float32)
        B32 = B.astype(np.float32)
        A32d, B32d = dev_cm(A32, torch), dev_cm(B32, torch)
        C32 = torch.empty_strided((N, N), (1, N), dtype=torch.float32, device="cuda")
        sms, sst = time_call(ozfp4, torch, lambda: ozfp4.sgemm(A32d, B32d, L32, out=C32),
                             max(3, args.steps // 2), 1)
        rows32 = np.arange(0, N, N // 64)[:64]
        ref32 = exact_reference(A32.astype(np.float64), B32.astype(np.float64), rows32, rows32)
        bits32, worst32 = accuracy_bits(block_of(C32, rows32, rows32, torch).astype(np.float64), ref32)
        Ar32, Br32 = torch.from_numpy(A32).to("cuda"), torch.from_numpy(B32).to("cuda")
        Cn32 = torch.matmul(Ar32, Br32)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(5):
            torch.matmul(Ar32, Br32, out=Cn32)
        torch.cuda.synchronize()
        nms32 = (time.perf_counter() - t0) * 1e3 / 5
        nbits32, nworst32 = accuracy_bits(block_of(Cn32, rows32, rows32, torch).astype(np.float64), ref32)
        flops32 = (4 * L32 - 1) * 2.0 * N ** 3
        one32 = None
        if not args.no_one_limb:
            # the one-limb list (11 first): the same 24-bit capacities with
            # 4 (L - 1) - 1 + 1 products; then the emulation with the three
            # lists and native FP32 timed alike, alternating
            L1 = one_limb(lambda: ozfp4.sgemm_moduli(N))
            oms32, ost32 = one_limb(lambda: time_call(
                ozfp4, torch, lambda: ozfp4.sgemm(A32d, B32d, L1, out=C32), max(3, args.steps // 2), 1))
            obits32, oworst32 = accuracy_bits(block_of(C32, rows32, rows32, torch).astype(np.float64),
                                              ref32)
            # three heads: the fewest limb products that reach the 24-bit
            # capacities at this k (11 moduli, 34 products)
            L3 = with_heads(3, lambda: ozfp4.sgemm_moduli(N))
            cap3 = list(with_heads(3, lambda: ozfp4.ozfp4_sgemm_capacity(N, L3)))
            C32g = torch.empty_like(C32)
            ozfp4.sgemm(A32d, B32d, L32, out=C32g)
            with_heads(3, lambda: ozfp4.sgemm(A32d, B32d, L3, out=C32))
            torch.cuda.synchronize()
            same3 = bool(torch.equal(C32.view(torch.int32), C32g.view(torch.int32)))
            del C32g
            calls32 = {"emulation": lambda: ozfp4.sgemm(A32d, B32d, L32, out=C32),
                       "emulation_one_limb": lambda: one_limb(lambda: ozfp4.sgemm(A32d, B32d, L1, out=C32)),
                       "emulation_three_heads": lambda: with_heads(
                           3, lambda: ozfp4.sgemm(A32d, B32d, L3, out=C32)),
                       "native_fp32": lambda: torch.matmul(Ar32, Br32, out=Cn32)}
            t32 = {k: stats(v) for k, v in paired_times(torch, calls32, max(5, args.steps // 2), 1).items()}
            one32 = {"n_moduli": L1, "capacity_bits": list(one_limb(lambda: ozfp4.ozfp4_sgemm_capacity(N, L1))),
                     "ms": oms32, "tflops": 2.0 * N ** 3 / oms32 / 1e9,
                     "stages_ms": dict(zip(stage_names, ost32)),
                     "products_per_element": 4 * (L1 - 1), "error_bits": obits32,
                     "max_normalized_error": oworst32,
                     "three_heads": {"n_moduli": L3, "capacity_bits": cap3,
                                     "products_per_element": 4 * L3 - 3 * 3 - 1,
                                     "c_bitwise_equal_to_greedy": same3},
                     "paired": {"protocol": "each call alone between synchronisations, HIP events, "
                                            "the four alternating", "ms": t32,
                                "one_limb_vs_native_fp32": t32["native_fp32"]["median"] /
                                t32["emulation_one_limb"]["median"],
                                "three_heads_vs_native_fp32": t32["native_fp32"]["median"] /
                                t32["emulation_three_heads"]["median"],
                                "greedy_vs_native_fp32": t32["native_fp32"]["median"] /
                                t32["emulation"]["median"]}}
        result["sgemm"] = {
            "workload": f"sgemm m=n=k={N}, phi=0.5 inputs rounded to FP32", "n_moduli": L32,
            "capacity_bits": list(ozfp4.ozfp4_sgemm_capacity(N, L32)), "ms": sms,
            "tflops": 2.0 * N ** 3 / sms / 1e9,
            "stages_ms": dict(zip(stage_names, sst)),
            "fp4_tflops_gemm": flops32 / sst[3] / 1e9,
            "error_bits": bits32, "max_normalized_error": worst32,
            "block": "64x64 (every 256th row and column)",
            "native_fp32": {"ms": nms32, "tflops": 2.0 * N ** 3 / nms32 / 1e9,
                            "error_bits": nbits32, "max_normalized_error": nworst32},
            "speedup_vs_native_fp32": nms32 / sms, "one_limb": one32}
        log(json.dumps(result["sgemm"]))
        del A32d, B32d, C32, Ar32, Br32, Cn32
        torch.cuda.empty_cache()

    if not args.no_int8:
        log("timing ozfp4_igemm_s8 8192^3")
        del Ad, Bd, C
        torch.cuda.empty_cache()
        A8, B8 = int8_inputs(8192, 8192, 8192, SEED + 40)
        A8d, B8d = dev_cm(A8, torch), dev_cm(B8, torch)
        C8 = torch.empty_strided((8192, 8192), (1, 8192), dtype=torch.int32, device="cuda")
        for _ in range(2):
            ozfp4.igemm_s8(A8d, B8d, out=C8)
        torch.cuda.synchronize()
        ozfp4.ozfp4_profile(True)
        reps = 5
        gsum = 0.0
        t0 = time.perf_counter()
        for _ in range(reps):
            ozfp4.igemm_s8(A8d, B8d, out=C8)
            gsum += ozfp4.ozfp4_stage_times()[2]
        torch.cuda.synchronize()
        ims = (time.perf_counter() - t0) * 1e3 / reps
        ozfp4.ozfp4_profile(False)
        gms = gsum / reps
        native8 = None
        try:
            # native INT8 matrix cores through torch (hipBLASLt), same inputs
            A8r = torch.from_numpy(A8).to("cuda")
            B8r = torch.from_numpy(np.ascontiguousarray(B8)).to("cuda")
            Cn8 = torch._int_mm(A8r, B8r)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(reps):
                torch._int_mm(A8r, B8r)
            torch.cuda.synchronize()
            nms8 = (time.perf_counter() - t0) * 1e3 / reps
            native8 = {"ms": nms8, "tops": 2.0 * 8192 ** 3 / nms8 / 1e9,
                       "c_bitwise_equal": bool(torch.equal(Cn8, C8))}
            del A8r, B8r, Cn8
        except Exception as err:  # noqa: BLE001 -- context only
            native8 = {"unavailable": str(err)[:200]}
        result["int8"] = {"workload": "igemm_s8 m=n=k=8192", "ms": ims,
                          "tops": 2.0 * 8192 ** 3 / ims / 1e9,
                          "gemm_ms": gms, "fp4_tflops_gemm": 9 * 2.0 * 8192 ** 3 / gms / 1e9,
                          "fp4_frac": 9 * 2.0 * 8192 ** 3 / gms / 1e9 / FP4_PEAK_TFLOPS,
                          "native_int8": native8}

    if not args.no_phi4:
        # the wide-dynamic-range workload: the paper's 53-bit cap with 19
        # moduli, and the wide-range extension (63 bits, 23 moduli)
        log("phi = 4 workload 8192 x 8192 x 32768")
        Ad = Bd = C = None
        torch.cuda.empty_cache()
        M4, K4 = 8192, 32768
        A4, B4 = dgemm_inputs(M4, M4, K4, 4.0, SEED + 4)
        A4d, B4d = dev_cm(A4, torch), dev_cm(B4, torch)
        C4 = torch.empty_strided((M4, M4), (1, M4), dtype=torch.float64, device="cuda")
        rows4 = np.arange(0, M4, M4 // 64)[:64]
        ref4 = exact_reference(A4, B4, rows4, rows4)
        runs = []
        for L4, cmax in ((19, 53), (23, 63)):
            ozfp4.ozfp4_set_max_capacity(cmax)
            try:
                ms4, st4 = time_dgemm(ozfp4, torch, A4d, B4d, C4, L4, 3, 1)
            finally:
                ozfp4.ozfp4_set_max_capacity(53)
            bits4, worst4 = accuracy_bits(block_of(C4, rows4, rows4, torch), ref4)
            runs.append({"route": "one-term conversion", "n_moduli": L4, "max_capacity": cmax,
                         "ms": ms4, "tflops": 2.0 * M4 * M4 * K4 / ms4 / 1e9, "gemm_ms": st4[3],
                         "error_bits": bits4, "max_normalized_error": worst4,
                         "fp64_accurate": worst4 <= 2.0 ** -50})
            log(json.dumps(runs[-1]))
        # the two-term split of the converted operands (19 moduli, the
        # paper's 53-bit capacities for both terms): four residue GEMMs
        ms4, st4 = time_call(ozfp4, torch, lambda: ozfp4.dgemm_split(A4d, B4d, 19, out=C4), 3, 1)
        C4b = block_of(C4, rows4, rows4, torch)
        bits4, worst4 = accuracy_bits(C4b, ref4)
        runs.append({"route": "two-term split", "n_moduli": 19, "max_capacity": 53, "ms": ms4,
                     "tflops": 2.0 * M4 * M4 * K4 / ms4 / 1e9, "gemm_ms": st4[3],
                     "stages_ms": dict(zip(["scale", "encode_A", "encode_B", "residue_gemms", "crt"], st4)),
                     "products_per_element": 4 * (4 * 19 - 1),
                     "error_bits": bits4, "max_normalized_error": worst4,
                     "fp64_accurate": worst4 <= 2.0 ** -50,
                     "vs_rounded_product": elementwise_vs_rounded(C4b, ref4)})
        log(json.dumps(runs[-1]))
        if not args.no_one_limb:
            # the same C from 21 moduli with the one-limb heads 11, 9, 8, 7
            # (the 19 greedy moduli's capacities at k = 32768)
            C4g = C4.clone()
            ms5, st5 = with_heads(4, lambda: time_call(
                ozfp4, torch, lambda: ozfp4.dgemm_split(A4d, B4d, 21, out=C4), 3, 1))
            runs.append({"route": "two-term split, 4 one-limb heads", "n_moduli": 21,
                         "max_capacity": 53, "ms": ms5,
                         "tflops": 2.0 * M4 * M4 * K4 / ms5 / 1e9, "gemm_ms": st5[3],
                         "products_per_element": 4 * (4 * 17 - 1 + 4),
                         "c_bitwise_equal_to_19_greedy_moduli": bool(
                             torch.equal(C4.view(torch.int64), C4g.view(torch.int64)))})
            log(json.dumps(runs[-1]))
            del C4g
        result["phi4"] = {"workload": "dgemm m=n=8192, k=32768, phi=4",
                          "block": "64x64 (every 128th row and column)", "runs": runs}
        del A4d, B4d, C4

    if cpu_rec is not None:
        result["cpu_baseline"] = cpu_rec

    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
