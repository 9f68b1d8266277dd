"""Host build of the two-term split's final step (paper_2608_06812_amd/
csrc/crt_split.hpp): X = X11 2^(2d) + X12 2^d + X22 in 256-bit two's
complement and one rounding of X 2^e2 to FP64, bit for bit against the
oracle's exact rounding of the same Python integer (RN(x 2^-shift), exact
rational arithmetic). Cases: the three products at their bounds with either
sign (k 2^106 for 53-bit capacities and k <= 2^16), heavy cancellation
between the terms, small values, exact ties and near-ties of the final
rounding, and scales that give subnormal results, underflow to zero and
overflow to infinity."""

import os
import random
import shutil
import struct
import subprocess

import pytest

import oracle as o

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "crt_split_host.cpp")
INC = os.path.join(ROOT, "paper_2608_06812_amd", "csrc")


@pytest.fixture(scope="module")
def split_bin(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no host C++ compiler")
    out = str(tmp_path_factory.mktemp("split") / "crt_split_host")
    subprocess.run([gxx, "-O2", "-std=c++17", "-I", INC, SRC, "-o", out], check=True)
    return out


def _words(x):
    m = abs(x)
    assert m < 1 << 192
    return f"{1 if x < 0 else 0} {m & (2**64 - 1):x} {(m >> 64) & (2**64 - 1):x} {m >> 128:x}"


def _cases(rng):
    out = []
    for _ in range(3000):
        d = rng.choice([1, 7, 30, 52, 53])
        k = rng.choice([1, 3, 1000, 1 << 16])
        big = k << 106
        x11 = rng.randint(-big, big)
        x12 = rng.randint(-big, big)
        x22 = rng.randint(-(k << 104), k << 104)
        X = (x11 << 2 * d) + (x12 << d) + x22
        e2 = rng.randint(-400, 0) - (X.bit_length() - 60 if X else 0) // 2
        out.append((d, e2, x11, x12, x22))
    for _ in range(1500):
        # cancellation: X12 2^d nearly cancels X11 2^2d
        d = rng.choice([20, 53])
        x11 = rng.randint(-(1 << 100), 1 << 100)
        x12 = -(x11 << d) + rng.randint(-(1 << 60), 1 << 60)
        x22 = rng.randint(-(1 << 90), 1 << 90)
        out.append((d, rng.randint(-200, 0), x11, x12, x22))
    for _ in range(1500):
        # small values, ties and near-ties: X = 2^p (odd) + half an ulp (+-1)
        d = rng.choice([5, 53])
        p = rng.randint(54, 200)
        base = (rng.getrandbits(53) | (1 << 52)) << (p - 52)
        tie = 1 << (p - 53)
        X = base + tie + rng.choice([-1, 0, 0, 1])
        x22 = X % (1 << d)
        rest = X >> d
        x12 = rest % (1 << d)
        x11 = rest >> d
        if rng.random() < 0.5:
            x11, x12, x22 = -x11, -x12, -x22
        out.append((d, rng.randint(-300, 100), x11, x12, x22))
    for e2 in (-1300, -1200, -1180, -1140, -1100, -1075, 700, 750, 800, 900):
        for _ in range(100):
            d = 53
            x11 = rng.randint(-(1 << 110), 1 << 110)
            out.append((d, e2, x11, rng.randint(-(1 << 100), 1 << 100), rng.randint(-(1 << 80), 1 << 80)))
    out.append((53, 0, 0, 0, 0))
    out.append((10, -5, 1, -(1 << 10), 0))      # exact zero from cancellation
    return out


def test_combination_and_rounding_bit_exact(split_bin):
    rng = random.Random(20261230)
    cases = _cases(rng)
    lines = "\n".join(f"{d} {e2} {_words(a)} {_words(b)} {_words(c)}" for d, e2, a, b, c in cases)
    res = subprocess.run([split_bin], input=lines + "\n", capture_output=True, text=True, check=True)
    got = res.stdout.split()
    assert len(got) == len(cases)
    for (d, e2, a, b, c), g in zip(cases, got):
        X = (a << 2 * d) + (b << d) + c
        want = o.round_scaled(X, -e2)
        wbits = struct.unpack("<Q", struct.pack("<d", want))[0]
        assert int(g, 16) == wbits, (d, e2, a, b, c)
