"""Build libtq.so (HIP for gfx950) in-tree.

    python paper_2607_16973_amd/build.py

Device code is compiled for gfx950 only, with packed-float32 instruction
selection disabled.  The two host-only solvers (codebook, rotation) are
plain C++ with OpenMP built by g++.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libtq.so")

HIP_SOURCES = ["encode.hip", "scan.hip", "batch.hip", "layout.hip", "calib.hip", "noalloc.hip",
               "api.cpp"]
# Per-source extra flags.  The scan's prefetch ring must stay where it is
# written: machine sinking would move every refill into the loop latch and
# serialise the loads with the table lookups (in the encode GEMM it moves
# the float64 folds out of the matrix-core stream and spills).  The atomic optimizer would
# turn the one-lane work-claim atomics into wave-wide ones whose result is
# read at once, stalling on the LDS round trip the scan hides.
EXTRA_FLAGS = {"encode.hip": ["-mllvm", "-disable-machine-sink"],
               "scan.hip": ["-mllvm", "-disable-machine-sink",
                            "-mllvm", "-amdgpu-atomic-optimizer-strategy=None"],
               "batch.hip": ["-mllvm", "-disable-machine-sink",
                             "-mllvm", "-amdgpu-atomic-optimizer-strategy=None"]}
HOST_SOURCES = ["codebook.cpp", "rotation.cpp"]


def _hipcc() -> str:
    for c in ("/opt/rocm/bin/hipcc", shutil.which("hipcc") or ""):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def hip_flags():
    return ["-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE, "-I", CSRC, "-Wno-unused-command-line-argument"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops" not in l and "is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError("build failed: %s\n%s" % (" ".join(cmd), out))
    return out


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    hipcc = _hipcc()
    jobs = []
    objs = []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        objs.append(obj)
        jobs.append([hipcc] + hip_flags() + EXTRA_FLAGS.get(src, []) +
                    ["-c", os.path.join(CSRC, src), "-o", obj])
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        objs.append(obj)
        jobs.append(["g++", "-O2", "-std=c++17", "-fPIC", "-fopenmp", "-I", INCLUDE, "-I", CSRC,
                     "-c", os.path.join(CSRC, src), "-o", obj])
    with ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        outs = list(ex.map(_run, jobs))
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    tmp = LIB + ".tmp%d" % os.getpid()
    _run([hipcc, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp] + objs + ["-lgomp"])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
