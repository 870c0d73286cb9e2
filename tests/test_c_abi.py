"""The C ABI from plain C: the header compiles as C11 (CPU), and a C program
linked against libkbfollow reproduces a hand-worked example on the GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c", "abi_check.c")


def test_header_is_plain_c(tmp_path):
    src = tmp_path / "h.c"
    src.write_text('#include "kbfollow.h"\nint main(void) { return KB_OK; }\n')
    subprocess.check_call(["gcc", "-std=c11", "-Wall", "-Werror", "-pedantic", "-fsyntax-only",
                           "-I", os.path.join(ROOT, "include"), str(src)])


def build_c_check(out_dir):
    import paper_2002_06115_amd as kbf
    exe = os.path.join(out_dir, "abi_check")
    libdir = os.path.dirname(kbf.LIB_PATH)
    subprocess.check_call(["gcc", "-std=c11", "-O1", "-D__HIP_PLATFORM_AMD__", "-I",
                           os.path.join(ROOT, "include"), "-I", "/opt/rocm/include", SRC,
                           "-o", exe, "-L", libdir, "-lkbfollow", "-L", "/opt/rocm/lib",
                           "-lamdhip64", f"-Wl,-rpath,{libdir}", "-Wl,-rpath,/opt/rocm/lib"])
    return exe


def test_c_program_builds(tmp_path):
    if not shutil.which("gcc") or not os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h"):
        pytest.skip("needs gcc and the ROCm headers")
    assert os.path.exists(build_c_check(str(tmp_path)))


@pytest.mark.gpu
def test_c_program_on_gpu(tmp_path):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    exe = build_c_check(str(tmp_path))
    out = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    assert "abi_check ok" in out.stdout
