"""Builds libkbfollow.so for gfx950 with hipcc (in-tree, no JIT cache).

Usage: ``python -m paper_2002_06115_amd.build`` or ``build()`` from Python.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT_DIR = os.path.join(PKG, "_lib")
LIB = os.path.join(OUT_DIR, "libkbfollow.so")
BUILD_DIR = os.path.join(PKG, "_build")

SOURCES = ["kernels.hip", "static_scratch.hip", "api.cpp", "plan.cpp"]

# Device code: gfx950 only.  Packed-FP32 instructions are disabled (the
# compiler would otherwise form v_pk_* from plain float code); no fast-math and
# no denormal flushing, so device arithmetic is plain IEEE.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
                "-packed-fp32-ops"]
COMMON_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-command-line-argument",
                "-I", INCLUDE]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libkbfollow)")


def build(verbose: bool = False, defines=(), out=None, build_dir=None, src_dir=None) -> str:
    """Compile and link the library; ``defines`` are extra -D flags (tuning
    experiments), ``out``/``build_dir``/``src_dir`` redirect inputs and outputs."""
    csrc = src_dir or CSRC
    out = out or LIB
    bdir = build_dir or BUILD_DIR
    os.makedirs(os.path.dirname(out), exist_ok=True)
    os.makedirs(bdir, exist_ok=True)
    extra = [f"-D{d}" for d in defines]
    cc = hipcc()
    objs = []
    for src in SOURCES:
        path = os.path.join(csrc, src)
        obj = os.path.join(bdir, src + ".o")
        if src.endswith(".hip"):
            cmd = [cc, "-x", "hip", *DEVICE_FLAGS, *COMMON_FLAGS, "-I", csrc, *extra, "-c", path,
                   "-o", obj]
        else:
            cmd = [cc, *COMMON_FLAGS, "-I", csrc, "-c", path, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
        objs.append(obj)
    tmp = out + ".tmp"
    cmd = [cc, *DEVICE_FLAGS, "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, out)
    fingerprint(defines, os.path.join(os.path.dirname(out), "kernels.fingerprint"), bdir, csrc)
    return out


CHECKED_LIB = os.path.join(OUT_DIR, "checked", "libkbfollow.so")


def build_checked(verbose: bool = False) -> str:
    """The follow library with in-kernel index validation (KBFOLLOW_CHECKED),
    for tests: every row, slot and combine index is checked before use and
    violations are counted (kb_checked_violations)."""
    return build(verbose, defines=("KBFOLLOW_CHECKED",), out=CHECKED_LIB,
                 build_dir=os.path.join(BUILD_DIR, "checked"))


def fingerprint(defines, path, bdir, csrc=CSRC) -> dict:
    """Per-kernel sha256 of the gfx950 assembly of kernels.hip, written as JSON
    {mangled kernel name: digest}: identifies the device code that rocprofv3
    counters were taken on (compiler-unique ids, debug lines and the numbering
    of basic-block labels, which depends on the kernel's place in the file,
    excluded)."""
    import hashlib
    import json
    import re
    asm = os.path.join(bdir, "kernels.s")
    cmd = [hipcc(), "-x", "hip", "--cuda-device-only", "-S", *DEVICE_FLAGS, *COMMON_FLAGS,
           "-I", csrc, *[f"-D{d}" for d in defines], os.path.join(csrc, "kernels.hip"), "-o", asm]
    subprocess.check_call(cmd, stderr=subprocess.DEVNULL)
    digests, name, h = {}, None, None
    start = re.compile(r"^(_Z\S+):\s*(;.*)?$")
    bb_label = re.compile(r"BB\d+_")  # .LBB<function>_<block>, also in comments
    with open(asm) as f:
        for line in f:
            m = start.match(line)
            if m and name is None:
                name, h = m.group(1), hashlib.sha256()
                continue
            if name is not None:
                if line.startswith(".Lfunc_end"):
                    digests[name] = h.hexdigest()
                    name = None
                elif "__hip_cuid" not in line and not line.lstrip().startswith((".loc", ".file")):
                    h.update(bb_label.sub("BB_", line).encode())
    with open(path, "w") as f:
        json.dump(digests, f, indent=0, sort_keys=True)
    return digests


CHAIN_LIB = os.path.join(OUT_DIR, "libkbchain.so")


def build_chain(verbose: bool = False) -> str:
    """Compile the multi-hop chain glue (include/kbchain.h) into its own
    shared library."""
    os.makedirs(OUT_DIR, exist_ok=True)
    tmp = CHAIN_LIB + ".tmp"
    cmd = [hipcc(), "-x", "hip", *DEVICE_FLAGS, *COMMON_FLAGS, "-shared",
           os.path.join(CSRC, "chain_glue.hip"), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, CHAIN_LIB)
    return CHAIN_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
    print(build_chain(verbose="-v" in sys.argv))
    print(build_checked(verbose="-v" in sys.argv))
