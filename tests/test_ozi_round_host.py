"""Host build of the library's scheme-I final reduction
(paper_2608_06812_amd/csrc/ozi_round.hpp, Sec. IV): x = sum_h 2197^h H_h
in 192-bit integers and one rounding RN(x 2^e2), checked bit for bit
against exact integer arithmetic and the oracle's rounding. Cases: random
partial sums of the size the GEMM produces, sums at the 2^131 bound the
reduction allows, cancellation to zero and to tiny values, exact ties, and
scale factors that give subnormal results, underflow and overflow."""

import os
import random
import shutil
import struct
import subprocess

import pytest

import oracle as o

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "ozi_round_host.cpp")
INC = os.path.join(ROOT, "paper_2608_06812_amd", "csrc")


@pytest.fixture(scope="module")
def red_bin(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no host C++ compiler")
    out = str(tmp_path_factory.mktemp("ozi") / "ozi_round_host")
    subprocess.run([gxx, "-O2", "-std=c++17", "-ffp-contract=fast", "-I", INC, SRC, "-o", out],
                   check=True)
    return out


def _compose(H):
    return sum(int(v) * 2197 ** h for h, v in enumerate(H))


def _cases(nh, rng):
    cases = []
    lim = 1 << 46     # partial sums of the GEMM stay below 2^45 for k <= 2^17
    for _ in range(800):
        cases.append(([rng.randint(-lim, lim) for _ in range(nh)], rng.randint(-2200, 40)))
    for _ in range(200):   # small magnitudes: leading groups zero
        H = [0] * nh
        H[rng.randrange(nh)] = rng.randint(-1000, 1000)
        H[0] = rng.randint(-(1 << 20), 1 << 20)
        cases.append((H, rng.randint(-1100, 10)))
    for _ in range(100):   # exact cancellation, then a tiny remainder
        H = [rng.randint(-lim, lim) for _ in range(nh)]
        if nh > 1:
            H[1] = rng.randint(-lim, lim)
            H[0] = -2197 * H[1] + rng.choice((0, 1, -1, 3))
            for h in range(2, nh):
                H[h] = 0
        cases.append((H, rng.randint(-60, 60)))
    for _ in range(100):   # near-ties of the final rounding
        x = (rng.randint(1 << 53, (1 << 54) - 1) | 1) << rng.randint(1, 40)
        H = []
        rest = x * rng.choice((1, -1))
        for _ in range(nh - 1):
            d = rest % 2197
            H.append(d)
            rest = (rest - d) // 2197
        H.append(rest)
        if abs(rest) < (1 << 62):
            cases.append((H, rng.randint(-1100, 900)))
    # both ends of the exponent range, and the largest magnitudes allowed
    top = min((1 << 130) // 2197 ** (nh - 1), (1 << 63) - 1)
    for e2 in (-2300, -1200, -1074 - 60, -1074, 0, 900, 1000, 1100):
        cases.append(([rng.randint(-lim, lim) for _ in range(nh)], e2))
        cases.append(([0] * (nh - 1) + [top], e2))
        cases.append(([0] * (nh - 1) + [-top], e2))
        cases.append(([rng.randint(-lim, lim) for _ in range(nh - 1)] + [top], e2))
    cases.append(([0] * nh, 0))
    return cases


@pytest.mark.parametrize("nh", [1, 3, 5, 9])
def test_ozi_reduction_matches_exact(red_bin, nh):
    rng = random.Random(500 + nh)
    cases = [(H, e2) for H, e2 in _cases(nh, rng) if abs(_compose(H)) < (1 << 131)]
    text = "".join(f"{nh} {e2} " + " ".join(map(str, H)) + "\n" for H, e2 in cases)
    res = subprocess.run([red_bin], input=text, capture_output=True, text=True, check=True)
    lines = res.stdout.split()
    assert len(lines) == len(cases)
    for (H, e2), got in zip(cases, lines):
        want = struct.unpack("<Q", struct.pack("<d", o.round_scaled(_compose(H), -e2)))[0]
        assert int(got, 16) == want, (H, e2)
