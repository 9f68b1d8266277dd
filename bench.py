"""Benchmark of the Ozaki-II-on-FP4 FP64 matrix product on one MI355X.

A step is one ozfp4_dgemm call on the m = n = k = 16384 workload (entries
(U(0,1) - 0.5) exp(0.5 N(0,1)), fixed seed, inputs resident in HBM): line
maxima and shifts, fused conversion + residues + limb encoding of A and of
B, the fused residue GEMM over all moduli, and the exact CRT
reconstruction. The printed JSON line carries the emulated-DGEMM rate
2 m n k / t, the residue GEMM against the FP4 matrix-core peak (stage time
measured with HIP events on the library's stream over the timed steps), the
CPU oracle timed on a bounded sample, a per-stage breakdown, native FP64
matrix product on the same GPU, Ozaki scheme I on the same limbs (checked
bit for bit against scheme II), the FP32 emulation beside native FP32 and
the INT8-on-FP4 path as context.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--moduli L]
                       [--size N] [--sweep] [--no-cpu-baseline] [--no-native] [--no-karatsuba]
                       [--no-phi4] [--no-ozi] [--no-sgemm] [--no-table1]
                       [--no-paper-accuracy]
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

# HBM bytes per launch of the residue GEMM at m = n = k = 16384, 18 moduli,
# from rocprofv3 FETCH_SIZE / WRITE_SIZE runs scaled by a 1 GiB copy
# (profiles/k_gemm_res_dgemm_16384_L18.md). Valid only for the GEMM source
# they were taken on, identified by the hash of its section of kernels.hpp.
MEASURED_TRAFFIC = {
    "kernel_source_sha256_16": "9bebb506c97596dd",
    "workload": (16384, 16384, 16384, 18),
    "read_GB": 154.6, "write_GB": 4.87,
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


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def dev_cm(X, torch):
    import numpy as np
    return torch.from_numpy(np.ascontiguousarray(X.T)).to("cuda").t()


def time_dgemm(ozfp4, torch, Ad, Bd, C, L, steps, warmup, profile=True):
    """Median-free protocol of the contract: W untimed calls, then K calls
    bracketed by synchronisations. Returns (ms per step, mean stage ms)."""
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


def cpu_baseline(A, B, L, k, budget_s=20.0):
    """The oracle, as it stands, on a bounded sample of output elements of
    the same workload (a square block of outputs, whole rows of A and
    columns of B at full k), grown until one timed run takes at least half
    of `budget_s` seconds (10-30 s of CPU work at the default), or reaches
    1024 x 1024."""
    import numpy as np

    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        blas_threads = 1
    side, elapsed, t64 = 64, 0.0, None
    while True:
        t0 = time.perf_counter()
        oracle.dgemm(A, B, L, rows=np.arange(side), cols=np.arange(side))
        elapsed = time.perf_counter() - t0
        t64 = elapsed if t64 is None else t64
        if elapsed >= budget_s / 2 or side >= 1024:
            break
        # cost grows between linearly and quadratically with the side
        side = min(1024, side * (2 if elapsed > budget_s / 8 else 4))
    tflops = 2.0 * k * side * side / elapsed / 1e12
    return {"value": tflops, "unit": "TFLOP/s (emulated DGEMM)", "cores": blas_threads,
            "kind": "oracle",
            "sample": f"{side}x{side} output block of the {A.shape[0]}x{B.shape[1]}x{k} workload at full k, "
                      f"{L} moduli, {elapsed:.2f} s (calibration 64x64: {t64:.2f} s); limb products "
                      f"in FP64 BLAS on {blas_threads} threads, exact CRT and rounding in "
                      f"single-threaded Python"}


def exact_reference(A, B, rows, cols):
    """Exact (AB)_ij and sum_k |A_ik||B_kj| on a block (oracle)."""
    import oracle
    return oracle.exact_block(A, B, rows, cols)


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


def block_of(C, rows, cols, torch):
    r = torch.as_tensor(rows, device="cuda")
    c = torch.as_tensor(cols, device="cuda")
    return C[r][:, c].cpu().numpy()


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=12)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--moduli", type=int, default=18)
    ap.add_argument("--size", type=int, default=16384)
    ap.add_argument("--sweep", action="store_true", help="sweep 12..20 moduli at the given size")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-native", action="store_true")
    ap.add_argument("--no-int8", action="store_true")
    ap.add_argument("--no-accuracy", action="store_true")
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
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this method has no multi-GPU path "
              "(its output tiles and moduli would shard without communication)",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2608_06812_amd import ozfp4
    from paper_2608_06812_amd.workloads import dgemm_inputs, int8_inputs, paper_law_inputs

    ozfp4.load()
    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    torch.cuda.set_device(0)
    N = args.size
    L = args.moduli

    log(f"generating inputs {N}^3")
    A, B = dgemm_inputs(N, N, N, 0.5, SEED + 2)
    Ad, Bd = dev_cm(A, torch), dev_cm(B, torch)
    C = torch.empty_strided((N, N), (1, N), dtype=torch.float64, device="cuda")

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
            bits, worst = accuracy_bits(block_of(C, rows, cols, torch), ref)
            rec = {"n_moduli": Ls, "ms": ms, "tflops": 2.0 * N ** 3 / ms / 1e9,
                   "gemm_ms": st[3], "error_bits": bits, "max_normalized_error": worst,
                   "fp64_accurate": worst <= 2.0 ** -50}
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
    flops_exec = (4 * L - 1) * 2.0 * N ** 3
    achieved = flops_exec / gemm_ms / 1e9
    stage_names = ["scale", "encode_A", "encode_B", "residue_gemm", "crt"]

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
    # runtime model t = 2 Q N^3 / R + D / beta (Eq. (model)) at the published peaks
    D = bytes_scale + 2 * bytes_enc + L * N * N + bytes_crt
    model_ms = (flops_exec / (FP4_PEAK_TFLOPS * 1e12) + D / (HBM_PEAK_GBS * 1e9)) * 1e3

    traffic = None
    if kernel_source_hash() == MEASURED_TRAFFIC["kernel_source_sha256_16"] and \
            (N, N, N, L) == MEASURED_TRAFFIC["workload"]:
        traffic = MEASURED_TRAFFIC["read_GB"] + MEASURED_TRAFFIC["write_GB"]

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
                     "traffic": traffic, "traffic_unit": "GB per launch (HBM read + write)",
                     "algorithmic_GB": (2 * L * N * N + L * N * N) / 1e9,
                     "flops_per_launch": flops_exec,
                     "avg_launch_ms": gemm_ms},
        "stages_ms": dict(zip(stage_names, stages)),
        "hbm_GBs": hbm,
        "model_ms": model_ms,
        "compute_stage_tflops": 2.0 * N ** 3 / (gemm_ms + stages[4]) / 1e9,
    }

    # the paper's runtime model with measured rates: beta from a plain 1 GiB
    # device copy (read + write bytes over time), R from the GEMM stage
    src = torch.empty(1 << 27, dtype=torch.float64, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    beta = 2.0 * src.numel() * 8 * 5 / (time.perf_counter() - t0) / 1e9
    result["hbm_copy_GBs"] = beta
    result["model_ms_measured"] = gemm_ms + D / (beta * 1e9) * 1e3
    del src, dst

    if args.copy_calibration:
        src = torch.empty(1 << 27, dtype=torch.float64, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = {"read": src.numel() * 8, "write": dst.numel() * 8}
        del src, dst

    ref_block = None
    if not args.no_accuracy:
        rows = np.arange(0, N, N // 128)[:128]
        cols = np.arange(0, N, N // 128)[:128]
        ref_block = exact_reference(A, B, rows, cols)
        bits, worst = accuracy_bits(block_of(C, rows, cols, torch), ref_block)
        result["accuracy"] = {"block": "128x128 (every N/128-th row and column)",
                              "error_bits": bits, "max_normalized_error": worst,
                              "fp64_accurate": worst <= 2.0 ** -50}

    if not args.no_native:
        log("timing native FP64 torch.matmul")
        Ar = torch.from_numpy(A).to("cuda")
        Br = torch.from_numpy(B).to("cuda")
        for _ in range(2):
            torch.matmul(Ar, Br)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        reps = 5
        for _ in range(reps):
            torch.matmul(Ar, Br)
        torch.cuda.synchronize()
        nms = (time.perf_counter() - t0) * 1e3 / reps
        result["native_fp64"] = {"ms": nms, "tflops": 2.0 * N ** 3 / nms / 1e9,
                                 "speedup_of_emulation": nms / ms}
        if ref_block is not None:
            # native FP64 accumulates rounding errors along k; same block
            Cn = torch.matmul(Ar, Br)
            nbits, nworst = accuracy_bits(block_of(Cn, rows, cols, torch), ref_block)
            result["native_fp64"].update({"error_bits": nbits, "max_normalized_error": nworst})
            del Cn
        del Ar, Br

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
            "speedup_vs_native_fp32": nms32 / sms}
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
            runs.append({"n_moduli": L4, "max_capacity": cmax, "ms": ms4,
                         "tflops": 2.0 * M4 * M4 * K4 / ms4 / 1e9, "gemm_ms": st4[3],
                         "error_bits": bits4, "max_normalized_error": worst4})
            log(json.dumps(runs[-1]))
        result["phi4"] = {"workload": "dgemm m=n=8192, k=32768, phi=4",
                          "block": "64x64 (every 128th row and column)", "runs": runs}
        del A4d, B4d, C4

    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline(A, B, L, N)

    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
