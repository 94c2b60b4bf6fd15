"""Build the CPU oracle (test infrastructure) into oracle/liboracle.so.

gcc, IEEE binary32 arithmetic: no FMA contraction, no fast-math, no
flush-to-zero.  OpenMP only spreads independent segments over threads.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "tco.c")
OUT = os.path.join(HERE, "liboracle.so")

CFLAGS = ["-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fno-finite-math-only",
          "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra", "-Wno-unused-function"]


# a checked build for the CPU test suite: address and undefined-behaviour
# sanitizers, any report fatal (host code only; the oracle has no GPU code)
SANITIZE = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
            "-fno-sanitize-recover=undefined"]


def build(verbose: bool = False, sanitize: bool = False, out: str | None = None) -> str:
    out = out or OUT
    tmp = out + ".tmp"
    cmd = ["gcc", *CFLAGS, *(SANITIZE if sanitize else []), SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
