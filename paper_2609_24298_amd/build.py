"""Build libkvc.so in-tree: host C++ with g++, HIP kernels with hipcc for gfx950.

Usage: python -m paper_2609_24298_amd.build
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
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libkvc.so")
ARCH = "gfx950"


def _hipcc() -> str:
    for c in ("/opt/rocm/bin/hipcc", shutil.which("hipcc") or ""):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libkvc)")


def _run(cmd):
    print("+", " ".join(cmd), flush=True)
    subprocess.check_call(cmd)


def build(verbose: bool = True) -> str:
    """Compile every source and link libkvc.so (always rebuilds)."""
    os.makedirs(BUILD, exist_ok=True)
    hipcc = _hipcc()
    host_o = os.path.join(BUILD, "kvc_host.o")
    _run(["g++", "-std=c++17", "-O2", "-fPIC", "-ffp-contract=off", "-fno-fast-math", "-Wall",
          "-I", INCLUDE, "-c", os.path.join(CSRC, "kvc_host.cpp"), "-o", host_o])
    objs = [host_o]
    # the HIP sources compile in parallel (the two decode partials units take most of the time)
    procs = []
    for src in ("kvc_decode_g4.hip", "kvc_decode_g8.hip", "kvc_decode.hip", "kvc_kernels.hip", "kvc_calib.hip"):
        o = os.path.join(BUILD, src.replace(".hip", ".o"))
        cmd = [hipcc, "-std=c++17", "-O3", "-fPIC", f"--offload-arch={ARCH}", "-ffp-contract=fast",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", o]
        print("+", " ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd)))
        objs.append(o)
    failed = [cmd for cmd, p in procs if p.wait() != 0]
    if failed:
        raise subprocess.CalledProcessError(1, failed[0])
    tmp = LIB + ".tmp%d" % os.getpid()
    _run([hipcc, "-shared", f"--offload-arch={ARCH}", "-o", tmp] + objs)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build()
    sys.exit(0)
