"""Compile libleyline.so and libleyline_exact.so (HIP kernels for gfx950 + the host planner) in-tree.

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
EXACT_LIB = os.path.join(HERE, "libleyline_exact.so")
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


def _start(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    return cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)


def _finish(job):
    cmd, proc = job
    out, _ = proc.communicate()
    if proc.returncode != 0:
        sys.stderr.write(out)
        raise RuntimeError(f"build step failed: {' '.join(cmd[:2])} ...")


def build(verbose: bool = False) -> str:
    """Both libraries, compiled side by side: libleyline.so (fp32 pair arithmetic) and
    libleyline_exact.so (fp64 pair arithmetic, LEYLINE_PAIR_F64=1)."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    os.makedirs(BUILD_DIR, exist_ok=True)
    inc = [f"-I{INCLUDE}", f"-I{CSRC}"]
    variants = [(LIB, "", []), (EXACT_LIB, "_exact", ["-DLEYLINE_PAIR_F64=1"])]
    jobs = []
    for _, tag, defs in variants:
        plan_o = os.path.join(BUILD_DIR, f"plan{tag}.o")
        kern_o = os.path.join(BUILD_DIR, f"kernels{tag}.o")
        jobs.append(_start(["g++", *HOST_FLAGS, *defs, *inc, "-c", os.path.join(CSRC, "plan.cpp"), "-o", plan_o], verbose))
        jobs.append(_start([hipcc, *HIP_FLAGS, *defs, *inc, "-c", os.path.join(CSRC, "kernels.hip"), "-o", kern_o], verbose))
    for job in jobs:
        _finish(job)
    for lib, tag, _ in variants:
        tmp = lib + ".tmp"
        _run([hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", os.path.join(BUILD_DIR, f"kernels{tag}.o"),
              os.path.join(BUILD_DIR, f"plan{tag}.o"), "-o", tmp], verbose)
        os.replace(tmp, lib)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
