"""The GEMM kernels' steady-state loops, checked in the gfx950 assembly of
this repository's own sources (hipcc -S, no GPU needed).

The streaming design relies on the compiler keeping a schedule: per stage a
fixed number of MFMAs, LDS reads and LDS-DMA copies (global or buffer
form), one barrier, no register spills, LDS reads issued several at a time
rather than each one waited for before its MFMA, and (residue, INT8,
scheme-I and Karatsuba GEMMs) every LDS read issued at least four MFMAs
before the wait for it. The compiler's schedule can change without any change
to a kernel's source (a change elsewhere in the translation unit is
enough); these checks catch a change of these properties before it
reaches the GPU."""

import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_06812_amd", "csrc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
         "-Xclang", "-packed-fp32-ops", "--cuda-device-only", "-S",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _hipcc():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cand = os.path.join(rocm, "bin", "hipcc")
    return cand if os.path.exists(cand) else shutil.which("hipcc")


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    hipcc = _hipcc()
    if hipcc is None:
        pytest.skip("no hipcc")
    out = {}
    d = tmp_path_factory.mktemp("asm")
    for tu in ("ozfp4.hip", "karatsuba.hip", "ozaki1.hip", "sgemm.hip", "split.hip",
               "calibrate.hip"):
        path = str(d / (tu + ".s"))
        subprocess.run([hipcc, *FLAGS, os.path.join(CSRC, tu), "-o", path], check=True,
                       capture_output=True)
        with open(path) as f:
            out[tu] = f.read()
    return out


def _function(text, mangled_prefix):
    lines = text.split("\n")
    body, on = [], False
    for line in lines:
        if not on and line.startswith(mangled_prefix) and line.split(";")[0].rstrip().endswith(":"):
            on = True
        if on:
            body.append(line)
            if line.strip().startswith(".Lfunc_end"):
                break
    assert body, mangled_prefix
    return body


def _loops(body):
    """Bodies of the loops closed by a backward conditional branch."""
    labels = {l.split(":")[0]: i for i, l in enumerate(body) if re.match(r"^\.LBB\d+_\d+:", l)}
    out = []
    for i, line in enumerate(body):
        m = re.search(r"s_cbranch_\w+\s+(\.LBB\d+_\d+)", line)
        if m and m.group(1) in labels and labels[m.group(1)] < i:
            out.append([x.strip() for x in body[labels[m.group(1)]:i + 1]
                        if x.startswith("\t") and not x.strip().startswith((";", "."))])
    return out


def _count(loop, pattern):
    return sum(1 for x in loop if re.search(pattern, x))


def _largest_read_batch(loop):
    """Largest number of LDS reads issued between two consecutive waits for
    all of them, going round the loop (a rotated loop may start with the
    wait for reads issued at the end of the previous iteration)."""
    full = [i for i, x in enumerate(loop) if x.startswith("s_waitcnt") and "lgkmcnt(0)" in x]
    if not full:
        return _count(loop, r"^ds_read")
    rot = loop[full[0] + 1:] + loop[:full[0] + 1]
    best = n = 0
    for x in rot:
        if x.startswith("ds_read"):
            n += 1
        elif x.startswith("s_waitcnt") and "lgkmcnt(0)" in x:
            best, n = max(best, n), 0
    return max(best, n)


def _min_read_cover(loop):
    """Fewest MFMAs the wave issues between an LDS read and the first wait
    that needs it done, going round the loop twice (the first pass only
    fills the queue of outstanding reads, which complete in order)."""
    pending, n_mfma, best = [], 0, None
    for lap in range(2):
        for x in loop:
            if x.startswith("ds_read"):
                pending.append(n_mfma)
            elif x.startswith("v_mfma"):
                n_mfma += 1
            elif x.startswith("s_waitcnt"):
                m = re.search(r"lgkmcnt\((\d+)\)", x)
                while m and len(pending) > int(m.group(1)):
                    cover = n_mfma - pending.pop(0)
                    if lap == 1:
                        best = cover if best is None else min(best, cover)
    return best


def test_no_kernel_spills(asm):
    for tu, text in asm.items():
        sizes = re.findall(r"\.set\s+(\S+)\.private_seg_size,\s*(\d+)", text)
        assert sizes, tu
        for name, size in sizes:
            assert int(size) == 0, (tu, name)


@pytest.mark.parametrize("tu,prefix,mfma,reads,dma", [
    ("ozfp4.hip", "_ZN5ozfp410k_gemm_res", 32, 16, 6),          # residue GEMM, k = 128 stage
    ("ozfp4.hip", "_ZN5ozfp49k_gemm_s8", 36, 18, 6),            # INT8 GEMM, k = 128 stage
    ("karatsuba.hip", "_ZN5ozfp414k_gemm_res_kar", 12, 12, 6),  # Karatsuba tile, k = 64 stage
    ("ozaki1.hip", "_ZN5ozfp410k_gemm_ozi", 36, 18, 6),         # scheme-I GEMM, k = 128 stage
])
def test_gemm_steady_loop(asm, tu, prefix, mfma, reads, dma):
    body = _function(asm[tu], prefix)
    loops = [l for l in _loops(body) if _count(l, r"v_mfma") == mfma]
    assert loops, f"no loop with {mfma} MFMAs in {prefix}"
    loop = loops[0]
    assert _count(loop, r"^ds_read_b128") == reads
    assert _count(loop, r"^(global_load_lds_dwordx4|buffer_load_dwordx4 .* lds$)") == dma
    assert _count(loop, r"^s_barrier") == 1
    assert _count(loop, r"scratch_") == 0
    # LDS reads go out in batches, several in flight before a wait for all
    assert _largest_read_batch(loop) >= 4, loop[:30]
    # every product is the unscaled FP4 form, which multiplies by 2^0: the
    # scaled form would take the scale operand the helper passes as byte 0
    # (E8M0 2^-127) at its face value
    assert _count(loop, r"^v_mfma_f32_32x32x64_f8f6f4 ") == mfma, loop[:30]
    assert _count(loop, r"v_mfma_scale|v_mfma_ld_scale") == 0


def test_no_scaled_mfma_anywhere(asm):
    """No kernel of the library issues a scaled MFMA form or loads a scale
    register: the E8M0 byte the helper passes is 0, which the scaled form
    would read as 2^-127."""
    for tu, text in asm.items():
        body = [x.strip() for x in text.split("\n") if x.startswith("\t")]
        assert _count(body, r"^v_mfma_scale|^v_mfma_ld_scale") == 0, tu
        if tu not in ("sgemm.hip", "split.hip"):   # these reuse the default GEMM
            assert _count(body, r"^v_mfma_f32_32x32x64_f8f6f4 ") > 0, tu


@pytest.mark.parametrize("tu,prefix,mfma", [
    ("ozfp4.hip", "_ZN5ozfp410k_gemm_res", 32),   # two-limb moduli
    ("ozfp4.hip", "_ZN5ozfp410k_gemm_res", 24),   # 169, without a1 b1
    ("ozfp4.hip", "_ZN5ozfp49k_gemm_s8", 36),     # three limbs (limb3_sched.hpp)
    ("ozaki1.hip", "_ZN5ozfp410k_gemm_ozi", 36),  # three limbs (limb3_sched.hpp)
    ("karatsuba.hip", "_ZN5ozfp414k_gemm_res_kar", 12),   # three-product tile
])
def test_gemm_reads_land_under_mfmas(asm, tu, prefix, mfma):
    """The GEMMs refill each operand register from LDS as soon as its last
    product group has been issued: every LDS read of the steady loop has at
    least four MFMAs of the wave between its issue and the wait for it, so
    the two waves of a SIMD do not stall on their reads together."""
    body = _function(asm[tu], prefix)
    loops = [l for l in _loops(body) if _count(l, r"v_mfma") == mfma]
    assert loops, f"no loop with {mfma} MFMAs"
    cover = _min_read_cover(loops[0])
    assert cover is not None and cover >= 4, cover
