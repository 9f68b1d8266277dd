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


def test_measured_traffic_matches_the_gemm_source():
    """The committed FETCH/WRITE figures belong to the residue GEMM source in
    the tree (bench.py prints them only while the hashes agree)."""
    assert bench.kernel_source_hash() == bench.MEASURED_TRAFFIC["kernel_source_sha256_16"]
    with open(os.path.join(ROOT, "profiles", "k_gemm_res_dgemm_16384_L18.md")) as f:
        text = f.read()
    assert "%.1f GB" % bench.MEASURED_TRAFFIC["read_GB"] in text
    assert "(%.2f GB)" % bench.MEASURED_TRAFFIC["write_GB"] in text


def test_cpu_baseline_record_on_a_tiny_workload():
    rng = np.random.default_rng(0)
    A = rng.random((64, 32)) - 0.5
    B = rng.random((32, 64)) - 0.5
    rec = bench.cpu_baseline(A, B, 14, 32, budget_s=0.01)
    assert rec["kind"] == "oracle" and rec["cores"] >= 1 and rec["value"] > 0
    assert "64x64" in rec["sample"]
    json.dumps(rec)


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
