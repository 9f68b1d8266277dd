"""The C ABI from plain C: tests/c_abi_client.c includes only
include/ozfp4.h and the HIP runtime's C API, links libozfp4.so, and checks
ozfp4_dgemm and ozfp4_igemm_s8 on small integer matrices against a CPU
triple loop (both products are exact integers). On the CPU the client is
compiled as C99 with warnings as errors and linked; on the GPU it runs as a
child process."""

import os
import shutil
import subprocess

import pytest

from paper_2608_06812_amd import ozfp4

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _build(out_dir):
    if not os.path.exists(ozfp4.LIB_PATH):
        from paper_2608_06812_amd import build
        build.build()
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    exe = os.path.join(str(out_dir), "c_abi_client")
    libdir = os.path.dirname(ozfp4.LIB_PATH)
    cmd = [cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
           os.path.join(ROOT, "tests", "c_abi_client.c"),
           "-L", libdir, "-lozfp4", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           f"-Wl,-rpath,{libdir}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    return exe


def test_c_client_compiles_and_links(tmp_path):
    exe = _build(tmp_path)
    assert os.path.exists(exe)


@pytest.mark.gpu
def test_c_client_runs(tmp_path):
    exe = _build(tmp_path)
    print("c_abi_client: dgemm 77x45x300 L=19, igemm_s8, dgemm_noalloc L=18, dgemm with 5 "
          "one-limb heads L=21, exact integers", flush=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.strip() == "OK"
