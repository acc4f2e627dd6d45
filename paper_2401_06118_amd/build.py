"""Build the HIP library ``libaqlm_mi355x.so`` for gfx950 with hipcc.

Each ``csrc/*.hip`` file compiles to an object in ``_build/`` (in parallel),
then one shared library is linked next to this file.  Packed fp32 VALU ops
are switched off for the device code (``-packed-fp32-ops``); hipcc's host
pass warns that it does not know that feature, which is harmless.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libaqlm_mi355x.so")
# Measurement-only microbenchmarks (bench.py --floors), a library of their own.
FLOORS_SRC = os.path.join(HERE, "floors", "floors.hip")
FLOORS_LIB = os.path.join(HERE, "libaqlm_floors.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["-std=c++17", "-O3", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-command-line-argument"]


# Per-file additions.  sorted.hip: one lane per workgroup takes a ticket with
# a returning atomic whose value is needed only at the end of the kernel; the
# atomic optimizer would aggregate it over the wave and read the result back
# at once, which stalls the wave for a memory round trip before its barrier.
FILE_FLAGS = {"sorted.hip": ["-mllvm", "-amdgpu-atomic-optimizer-strategy=None"]}


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.basename(src)[:-4] + ".o")
    cmd = [HIPCC, *FLAGS, *FILE_FLAGS.get(os.path.basename(src), []), "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{out}")
    if out and verbose:
        print(out)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    tmp = FLOORS_LIB + ".tmp"
    cmd = [HIPCC, *FLAGS, "-shared", "-o", tmp, FLOORS_SRC]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {FLOORS_SRC}:\n{r.stdout}{r.stderr}")
    os.replace(tmp, FLOORS_LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
