"""Compile libleyline.so (HIP kernels for gfx950 + the host planner) in-tree.

Usage: python -m paper_2606_01065_amd.build   (always recompiles)
"""

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libleyline.so")
BUILD_DIR = os.path.join(HERE, "_build")

ARCH = "gfx950"
HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # packed fp32 vector ops are disabled for all device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd[:2])} ...")
    return res


def build(verbose: bool = False) -> str:
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    os.makedirs(BUILD_DIR, exist_ok=True)
    inc = [f"-I{INCLUDE}", f"-I{CSRC}"]
    plan_o = os.path.join(BUILD_DIR, "plan.o")
    kern_o = os.path.join(BUILD_DIR, "kernels.o")
    _run(["g++", *HOST_FLAGS, *inc, "-c", os.path.join(CSRC, "plan.cpp"), "-o", plan_o], verbose)
    _run([hipcc, *HIP_FLAGS, *inc, "-c", os.path.join(CSRC, "kernels.hip"), "-o", kern_o], verbose)
    tmp = LIB + ".tmp"
    _run([hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", kern_o, plan_o, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
