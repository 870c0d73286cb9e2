"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The layout planner behind kb_create (paper_2002_06115_amd/csrc/plan.cpp, pure
host C++) and the CPU oracle (oracle/kb_oracle.c) are built with
-fsanitize=address,undefined by the host compilers and driven by the
programs under tests/c/, which also check the plan's invariants and the
oracle's entry points against each other.  No GPU code is involved.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2002_06115_amd", "csrc")
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer"]


def run_sanitized(exe):
    env = dict(os.environ, ASAN_OPTIONS="verify_asan_link_order=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    if r.returncode != 0 and "LeakSanitizer has encountered a fatal error" in r.stderr:
        # Leak checking cannot run in this environment (ptrace): keep the rest.
        env["ASAN_OPTIONS"] += ":detect_leaks=0"
        r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    return r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_planner_under_sanitizers(tmp_path):
    exe = str(tmp_path / "plan_sanitized")
    subprocess.check_call(["g++", "-std=c++17", *SAN, "-I", CSRC,
                           os.path.join(ROOT, "tests", "c", "plan_sanitized.cpp"),
                           os.path.join(CSRC, "plan.cpp"), "-o", exe])
    assert "planner checks passed" in run_sanitized(exe)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_sanitized")
    subprocess.check_call(["gcc", "-std=c11", "-fopenmp", *SAN,
                           os.path.join(ROOT, "tests", "c", "oracle_sanitized.c"),
                           os.path.join(ROOT, "oracle", "kb_oracle.c"), "-o", exe, "-lm"])
    assert "oracle checks passed" in run_sanitized(exe)
