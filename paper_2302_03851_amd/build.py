"""Build libedb.so (host library + gfx950 kernels) in-tree.

    python -m paper_2302_03851_amd.build

Host C++ parts are compiled with g++, the HIP parts with hipcc for gfx950;
the shared library lands next to this file.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libedb.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")

HOST_SRC = ["graph.cpp", "schedule.cpp", "learn.cpp", "plan.cpp", "pqplan.cpp", "forward.cpp"]
HIP_SRC = ["exec.hip", "diag.hip"]

# -ffp-contract=off: the policy learner's floating-point updates round as written
CXXFLAGS = ["-O2", "-fPIC", "-std=c++17", "-Wall", "-ffp-contract=off", "-I", os.path.join(ROOT, "include")]
# Packed fp32 instructions are disabled for all device code.
# -ffp-contract=off: every kernel rounds the same expression the same way
# (fused multiply-adds are written out where they are wanted), which keeps
# results bitwise equal across tile variants.
HIPFLAGS = ["-O3", "-fPIC", "-std=c++17", "--offload-arch=gfx950", "-ffp-contract=off",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(" ".join(cmd) + "\n" + r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {cmd[0]} {cmd[-1]}")
    return r


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = []
    objs = []
    for f in HOST_SRC:
        o = os.path.join(BUILD, f + ".o")
        jobs.append(["g++", *CXXFLAGS, "-c", os.path.join(CSRC, f), "-o", o])
        objs.append(o)
    for f in HIP_SRC:
        o = os.path.join(BUILD, f + ".o")
        jobs.append([HIPCC, *HIPFLAGS, "-c", os.path.join(CSRC, f), "-o", o])
        objs.append(o)
    with ThreadPoolExecutor(max_workers=4) as ex:
        list(ex.map(_run, jobs))
    tmp = LIB + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
