"""Builds libozfp4.so (gfx950) in the package directory with hipcc.

Usage: python -m paper_2608_06812_amd.build   (or build() from Python)
"""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libozfp4.so")
# seven translation units: the API with the default kernels, the Karatsuba
# mode's kernels, the scheme-I kernels, the FP32-emulation kernels, the
# two-term split's kernels, the one-limb modulus's GEMM and the
# reference-measurement kernels (kept apart so they cannot change the
# default kernels' code)
SOURCES = [os.path.join(HERE, "csrc", n)
           for n in ("ozfp4.hip", "karatsuba.hip", "ozaki1.hip", "sgemm.hip", "split.hip",
                     "onelimb.hip", "calibrate.hip")]
HEADERS = [os.path.join(HERE, "csrc", n) for n in
           ("device_common.hpp", "kernels.hpp", "karatsuba.hpp", "crt_round.hpp", "tables.hpp",
            "ozaki1.hpp", "ozi_round.hpp", "sgemm.hpp", "crt_round_f32.hpp",
            "calibrate.hpp", "split.hpp", "crt_split.hpp", "onelimb.hpp", "plain_gemm.hpp", "limb3_sched.hpp")] + \
          [os.path.join(ROOT, "include", "ozfp4.h")]

# -packed-fp32-ops: keep the compiler from emitting packed FP32 arithmetic.
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cand = os.path.join(rocm, "bin", "hipcc")
    return cand if os.path.exists(cand) else "hipcc"


def build(verbose: bool = False) -> str:
    """Compile the library; returns its path. Always recompiles."""
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *FLAGS, "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc"),
           *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed to build libozfp4.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
