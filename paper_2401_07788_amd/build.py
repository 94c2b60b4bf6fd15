"""Build libtc.so (the gfx950 HIP library) in-tree with hipcc.

Every translation unit is compiled for gfx950 only, with IEEE binary32
arithmetic (no FMA contraction, denormals kept) and without packed-fp32
instruction selection, then linked into one shared library that exports the
C ABI of include/tc.h and nothing else.

libtc_debug.so is the same library with the C-ABI layer compiled with
TC_DEBUG: before each launch it checks the preconditions the release library
assumes (finite inputs, distinct AQ-SGD ids, no overlapping buffers) and
returns TC_ERR_PRECONDITION when one fails; the check kernels of k_check.hip
are linked into it only.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libtc.so")
LIB_DEBUG = os.path.join(HERE, "libtc_debug.so")
KERNELS = ["k_topk.hip", "k_quant.hip", "k_scatter.hip", "k_global.hip", "k_scratch.hip"]
API = "tc_api.cpp"
CHECKS = "k_check.hip"
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", "-ffp-contract=off", "-fvisibility=hidden", "-Wall",
          "-Wno-unused-function"]
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc():
    for p in ("/opt/rocm/bin/hipcc", "hipcc"):
        if os.path.sep not in p or os.path.exists(p):
            return p
    return "hipcc"


def _compile(src: str, verbose: bool, debug: bool = False) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ("_debug" if debug else "") + ".o")
    cmd = [_hipcc(), *COMMON]
    if debug:
        cmd += ["-DTC_DEBUG"]
    if src.endswith(".hip"):
        cmd += ["-x", "hip", *DEVICE]
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def _link(objs, lib: str, verbose: bool):
    tmp = lib + ".tmp"
    cmd = [_hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)


def build(verbose: bool = False, jobs: int | None = None) -> str:
    os.makedirs(BUILD, exist_ok=True)
    units = [(s, False) for s in KERNELS + [API, CHECKS]] + [(API, True)]
    jobs = jobs or min(len(units), max(1, (os.cpu_count() or 2)))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = dict(zip(units, ex.map(lambda u: _compile(u[0], verbose, u[1]), units)))
    kernels = [objs[(s, False)] for s in KERNELS]
    _link(kernels + [objs[(API, False)]], LIB, verbose)
    _link(kernels + [objs[(CHECKS, False)], objs[(API, True)]], LIB_DEBUG, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
