"""Build libewsjf.so (the HIP library behind include/ewsjf.h) for gfx950.

Every translation unit is compiled with hipcc for gfx950 only, without
floating-point contraction (the partitioner's binary64 arithmetic must match
its definition exactly) and without packed fp32 instructions.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INC = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libewsjf.so")
BUILD = os.path.join(PKG, "_build")
# The instrumented variant (phase stamps, read by phase_stamps.py).
LIB_STAMPS = os.path.join(PKG, "libewsjf_stamps.so")
BUILD_STAMPS = os.path.join(PKG, "_build_stamps")
SOURCES = ["abi.hip", "kern_policy.hip", "kern_select.hip", "kern_partition.hip", "kern_tactical.hip",
           "kern_dispatch.hip", "kern_trial.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-result", "-I", INC, "-I", CSRC]


def _compile(src: str, verbose: bool, stamps: bool = False) -> str:
    obj = os.path.join(BUILD_STAMPS if stamps else BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *(["-DEWSJF_STAMPS"] if stamps else []), "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{msg}")
    if verbose and msg.strip():
        print(msg, flush=True)
    return obj


def build(verbose: bool = False, stamps: bool = False) -> str:
    """Build libewsjf.so, or with stamps=True the instrumented
    libewsjf_stamps.so (same kernels plus phase timestamps)."""
    lib = LIB_STAMPS if stamps else LIB
    os.makedirs(BUILD_STAMPS if stamps else BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, stamps), SOURCES))
    tmp = lib + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, stamps="--stamps" in sys.argv))
