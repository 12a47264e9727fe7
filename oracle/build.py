"""Build the CPU oracle shared library (test infrastructure only).

g++ -O2 -ffp-contract=off keeps every binary64 operation as written.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ewsjf_oracle.cpp")
LIB = os.path.join(HERE, "libewsjf_oracle.so")


def build(verbose: bool = False, sanitize: bool = False, out: str | None = None) -> str:
    out = out or LIB
    cmd = ["g++", "-std=c++17", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
           "-Wall", "-Wextra", SRC, "-o", out + ".tmp"]
    if sanitize:
        cmd[3:3] = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-g"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    build(verbose=True, sanitize="--sanitize" in sys.argv)
