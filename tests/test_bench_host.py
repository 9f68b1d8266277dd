"""Host-side checks of bench.py that need no GPU: the one-GPU contract, the
guard that ties the committed HBM byte counters to the GEMM source they
were taken on, and the CPU-baseline and accuracy helpers on tiny inputs."""

import json
import os
import subprocess
import sys

import numpy as np

import oracle as o

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""


def test_measured_traffic_is_tied_to_the_gemm_source(monkeypatch):
    """bench.py reports the committed FETCH/WRITE figures only for the
    residue-GEMM source and workload they were taken on; when they are
    committed, the profile summary holds the same raw counters."""
    t = dict(bench.MEASURED_TRAFFIC)
    if t["kernel_source_sha256_16"] is not None:
        with open(os.path.join(ROOT, t["profile"])) as f:
            text = f.read()
        assert f"{t['fetch_kib']:,}" in text and f"{t['write_kib']:,}" in text
        assert t["kernel_source_sha256_16"] in text
        if t["kernel_source_sha256_16"] == bench.kernel_source_hash():
            got = bench.measured_traffic(*t["workload"][2:])
            assert got is not None and got["fetch_size_kib_raw"] == t["fetch_kib"]
    fake = dict(t, kernel_source_sha256_16=bench.kernel_source_hash(), fetch_kib=1000,
                write_kib=10, fetch_factor=2.0, write_factor=1.0)
    monkeypatch.setattr(bench, "MEASURED_TRAFFIC", fake)
    got = bench.measured_traffic(16384, 18)
    assert abs(got["GB"] - (1000 * 1024 * 2.0 + 10 * 1024) / 1e9) < 1e-12
    assert bench.measured_traffic(8192, 18) is None            # another workload
    monkeypatch.setattr(bench, "MEASURED_TRAFFIC", dict(fake, kernel_source_sha256_16="0" * 16))
    assert bench.measured_traffic(16384, 18) is None           # another source


def test_cpu_baseline_record_on_a_tiny_workload():
    rng = np.random.default_rng(0)
    A = rng.random((64, 32)) - 0.5
    B = rng.random((32, 64)) - 0.5
    rec = bench.cpu_baseline(A, B, 14, 32, budget_s=0.01)
    assert rec["kind"] == "oracle" and rec["cores"] >= 1 and rec["value"] > 0
    assert "64x64" in rec["sample"] and rec["os_cpu_count"] == os.cpu_count()
    json.dumps(rec)


def test_cpu_baseline_pool_covers_the_block():
    """With several workers and a block of several tiles, every output of
    the block is computed once (tiles of 256 x 256)."""
    rng = np.random.default_rng(5)
    A = rng.random((600, 40)) - 0.5
    B = rng.random((40, 600)) - 0.5
    rec = bench.cpu_baseline(A, B, 14, 40, budget_s=1e9, workers=3, max_side=512)
    assert rec["cores"] == 3 and "512x512" in rec["sample"]


def test_elementwise_metric_against_the_rounded_product():
    rng = np.random.default_rng(2)
    A = rng.random((3, 30)) - 0.5
    B = rng.random((30, 4)) - 0.5
    rows, cols = np.arange(3), np.arange(4)
    ref = bench.exact_reference(A, B, rows, cols)
    fl = np.array([[float(ref[0][i, j]) for j in range(4)] for i in range(3)])
    rec = bench.elementwise_vs_rounded(fl, ref)
    assert rec["max_rel_error"] == 0.0 and rec["frac_equal_to_fl"] == 1.0 and rec["max_ulps"] == 0
    off = fl.copy()
    off[1, 2] = np.nextafter(off[1, 2], np.inf)
    rec = bench.elementwise_vs_rounded(off, ref)
    assert rec["max_ulps"] == 1 and rec["frac_equal_to_fl"] == 11 / 12
    assert 0 < rec["max_rel_error"] <= 2.0 ** -52 and rec["frac_within_2^-50"] == 1.0


def test_stats():
    st = bench.stats([3.0, 1.0, 2.0, 10.0])
    assert st["median"] == 2.5 and st["min"] == 1.0 and st["max"] == 10.0 and st["n"] == 4


def test_accuracy_bits_against_the_exact_block():
    rng = np.random.default_rng(1)
    A = rng.random((4, 20)) - 0.5
    B = rng.random((20, 3)) - 0.5
    rows, cols = np.arange(4), np.arange(3)
    ref = bench.exact_reference(A, B, rows, cols)
    C = o.dgemm(A, B, 18)["C"]
    bits, worst = bench.accuracy_bits(C, ref)
    assert bits >= 52 and worst <= 2.0 ** -52
    bits_native, _ = bench.accuracy_bits((A.astype(np.float32) @ B.astype(np.float32)).astype(np.float64), ref)
    assert bits_native < bits


def test_source_hash_ignores_comments_but_not_code():
    code = "int f(int x) {\n  // a comment\n  return x + 1; /* another */\n}\n"
    assert bench.code_only(code) == bench.code_only(code.replace("a comment", "edited"))
    assert bench.code_only(code) == bench.code_only(code.replace("\n  ", "\n    "))
    assert bench.code_only(code) != bench.code_only(code.replace("x + 1", "x + 2"))
    assert "comment" not in bench.code_only(code) and "another" not in bench.code_only(code)


def test_exact_reference_against_fractions():
    """bench.py's own exact block product (it does not use the oracle)
    against plain Fraction sums, on entries spread over many binades, zeros
    and negative values included."""
    from fractions import Fraction
    rng = np.random.default_rng(9)
    A = (rng.random((5, 37)) - 0.5) * np.exp2(rng.integers(-60, 60, (5, 37)))
    B = (rng.random((37, 4)) - 0.5) * np.exp2(rng.integers(-60, 60, (37, 4)))
    A[1, :] = 0.0
    A[2, 3] = 5e-320                     # subnormal
    B[7, 2] = -0.0
    rows, cols = np.array([0, 1, 2, 4]), np.array([0, 2, 3])
    ex, ab = bench.exact_reference(A, B, rows, cols)
    for a, i in enumerate(rows):
        for b, j in enumerate(cols):
            want = sum(Fraction(float(A[i, q])) * Fraction(float(B[q, j])) for q in range(37))
            wabs = sum(abs(Fraction(float(A[i, q])) * Fraction(float(B[q, j]))) for q in range(37))
            assert ex[a, b] == want and ab[a, b] == wabs
    # and the oracle's independent block product agrees
    oe, oa = o.exact_block(A, B, rows, cols)
    assert np.all(oe == ex) and np.all(oa == ab)
