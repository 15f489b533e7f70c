"""Build libhuge2.so in-tree with hipcc for gfx950.

Run as ``python -m paper_1907_11210_amd._build`` or through
``__graft_entry__.build()``.  Compiles every source under ``csrc/`` each time
it is called.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libhuge2.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["plan.cpp", "capi.cpp", "kernels.hip"]

# Packed-FP32 VALU ops are disabled for all device code; the host pass only
# warns that it does not know the feature.  MFMA accumulators live in
# ordinary VGPRs (-amdgpu-mfma-vgpr-form): kernels whose accumulators the
# compiler would place in AGPRs then skip the copies to and from them in
# every epilogue (the column-phase kernel's tile epilogues spent 32 of their
# VALU instructions on those copies), and no kernel needs more registers.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
                "-packed-fp32-ops", "-mllvm", "-amdgpu-mfma-vgpr-form"]
COMMON_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-I", os.path.join(ROOT, "include"),
                "-I", CSRC]


def build(verbose: bool = False) -> str:
    build_dir = os.path.join(PKG, "_build")
    os.makedirs(build_dir, exist_ok=True)
    procs, objs = [], []
    for src in SOURCES:  # the translation units compile in parallel
        path = os.path.join(CSRC, src)
        obj = os.path.join(build_dir, src + ".o")
        cmd = [HIPCC] + COMMON_FLAGS + DEVICE_FLAGS + ["-x", "hip", "-c", path, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd)))
        objs.append(obj)
    failed = [cmd for cmd, p in procs if p.wait() != 0]
    if failed:
        raise subprocess.CalledProcessError(1, failed[0])
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "-shared", "-fPIC"] + DEVICE_FLAGS + objs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
