"""Build librs.so (HIP kernels for gfx950 + host C ABI) in-tree.

    python -m paper_2608_29058_amd.build [-j N]

Each HIP translation unit is compiled with hipcc for gfx950 only; the host router is plain
C++ and, like the device router, is compiled with floating-point contraction disabled (its
fp64 operation order is part of its definition).
"""
from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "librs.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")

HIP_SOURCES = ["attn.hip", "probe.hip", "topk.hip", "route_dev.hip"]
# sources whose fp64 operation order is part of their definition
NO_CONTRACT = {"route_dev.hip"}
HOST_HIP_SOURCES = ["api.cpp"]
PLAIN_SOURCES = ["route.cpp"]

HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-munsafe-fp-atomics", "-Wno-unused-result"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(" ".join(cmd) + "\n" + r.stdout + r.stderr)
        raise RuntimeError(f"compile failed: {cmd[-3] if len(cmd) > 3 else cmd}")
    return r


def build(jobs: int | None = None, verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    cmds = []
    objs = []
    for s in HIP_SOURCES:
        o = os.path.join(BUILD, s + ".o")
        extra = ["-ffp-contract=off"] if s in NO_CONTRACT else []
        cmds.append([HIPCC, *HIP_FLAGS, *extra, "-c", os.path.join(CSRC, s), "-o", o])
        objs.append(o)
    for s in HOST_HIP_SOURCES:
        o = os.path.join(BUILD, s + ".o")
        cmds.append([HIPCC, "-O2", "-fPIC", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-c",
                     os.path.join(CSRC, s), "-o", o])
        objs.append(o)
    cxx = shutil.which("g++") or "g++"
    for s in PLAIN_SOURCES:
        o = os.path.join(BUILD, s + ".o")
        cmds.append([cxx, "-O2", "-fPIC", "-std=c++17", "-ffp-contract=off", "-c",
                     os.path.join(CSRC, s), "-o", o])
        objs.append(o)
    jobs = jobs or min(len(cmds), os.cpu_count() or 1)
    with ThreadPoolExecutor(jobs) as ex:
        for r in ex.map(_run, cmds):
            if verbose and (r.stdout or r.stderr):
                sys.stderr.write(r.stdout + r.stderr)
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("-j", type=int, default=None)
    ap.add_argument("-v", action="store_true")
    a = ap.parse_args()
    print(build(a.j, a.v))
