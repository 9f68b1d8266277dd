"""Host build of the library's CRT reconstruction and final rounding
(paper_2608_06812_amd/csrc/crt_round.hpp, Sec. V-B), checked bit for bit
against the oracle's exact symmetric CRT and RN(x 2^-shift) (exact rational
arithmetic). Both the FP64 fast path and the exact 192-bit path are
checked on every case. The cases cover uniform residues, small values, the
boundaries of the fast path's two branches (|t| = 2, 3 at chunk 2^84),
exact ties and near-ties of the final rounding, +-P/2, and scale factors
that give subnormal results, underflow to zero and overflow to infinity.
The binary32 rounding of the FP32 emulation (crt_round_f32.hpp) is checked
on the same cases against the oracle's exact binary32 rounding."""

import math
import os
import random
import shutil
import struct
import subprocess

import pytest

import oracle as o

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "crt_round_host.cpp")
INC = os.path.join(ROOT, "paper_2608_06812_amd", "csrc")


@pytest.fixture(scope="module")
def crt_bin(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no host C++ compiler")
    out = str(tmp_path_factory.mktemp("crt") / "crt_round_host")
    # contraction on, as in the device build
    subprocess.run([gxx, "-O2", "-std=c++17", "-ffp-contract=fast", "-I", INC, SRC, "-o", out],
                   check=True)
    return out


def _cases(L, rng):
    ms = o.select_moduli(L)
    P = math.prod(ms)
    half = P // 2
    lo = -half + (1 if P % 2 == 0 else 0)     # symmetric range (-P/2, P/2]
    xs = []
    for _ in range(1500):
        xs.append((rng.randint(lo, half), rng.randint(-200, 200)))
    for _ in range(600):
        b = rng.randint(0, min(90, P.bit_length() - 2))
        xs.append((rng.choice((-1, 1)) * rng.randint(0, 1 << b), rng.randint(-100, 100)))
    for t in range(-5, 6):
        for _ in range(20):
            x = t * (1 << 84) + rng.randint(0, (1 << 84) - 1)
            if lo <= x <= half:
                xs.append((x, rng.randint(-50, 50)))
    if P.bit_length() > 60:
        for _ in range(800):
            E = rng.randint(54, P.bit_length() - 2)
            mant = rng.randint(1 << 52, (1 << 53) - 1)
            x = ((2 * mant + 1) << (E - 53)) + rng.choice((0, 0, 1, -1, 2, -2))
            x *= rng.choice((-1, 1))
            if lo <= x <= half:
                xs.append((x, rng.randint(-30, 30)))
    for _ in range(400):   # near-ties of the binary32 rounding
        E = rng.randint(25, max(25, P.bit_length() - 2))
        mant = rng.randint(1 << 23, (1 << 24) - 1)
        x = ((2 * mant + 1) << (E - 24)) + rng.choice((0, 0, 1, -1, 2, -2))
        x *= rng.choice((-1, 1))
        if lo <= x <= half:
            xs.append((x, rng.randint(-30, 30)))
    for x in (half, lo, half - 1, lo + 1, 0, 1, -1, (1 << 53) - 1, 1 << 53, (1 << 53) + 1):
        if lo <= x <= half:
            for e2 in (0, -1204, -1100, -1082, -1140, 900, 1000, 923, -2000, 2000,
                       -149, -150, -172, -180, 104, 127, 128):
                xs.append((x, e2))
    for _ in range(150):
        x = rng.randint(lo, half)
        n = max(x.bit_length(), 1)
        xs.append((x, rng.choice((-1074 - n + rng.randint(0, 60), 1024 - n + rng.randint(-3, 3)))))
    return [(x, e2, [x % m for m in ms]) for x, e2 in xs]


@pytest.mark.parametrize("L", [2, 9, 14, 17, 18, 19, 20, 23, 27])
def test_crt_round_matches_exact_rational(crt_bin, L):
    rng = random.Random(1000 + L)
    cases = _cases(L, rng)
    text = "".join(f"{L} {e2} " + " ".join(map(str, r)) + "\n" for _, e2, r in cases)
    res = subprocess.run([crt_bin], input=text, capture_output=True, text=True, check=True)
    lines = res.stdout.split("\n")
    fast_count = fast32_count = 0
    for (x, e2, r), line in zip(cases, lines):
        got, exact, fast, f32, f32fast, fast32 = line.split()
        want = struct.unpack("<Q", struct.pack("<d", o.round_scaled(x, -e2)))[0]
        assert int(exact, 16) == want, (L, x, e2, "exact path")
        assert int(got, 16) == want, (L, x, e2, "fast path" if fast == "1" else "exact path")
        want32 = int(o.round_scaled_f32(x, -e2).view("uint32"))
        assert int(f32, 16) == want32, (L, x, e2, "binary32")
        if fast32 == "1":
            assert int(f32fast, 16) == want32, (L, x, e2, "binary32 fast path")
        fast_count += int(fast)
        fast32_count += int(fast32)
    assert len(lines) >= len(cases)
    if L <= 19:   # three chunks: most elements take the fast paths
        assert fast_count > 0.8 * len(cases) and fast32_count > 0.8 * len(cases)
    else:
        assert fast_count == 0 and fast32_count == 0
