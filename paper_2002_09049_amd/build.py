"""Compile the HIP library libmpq.so for gfx950 in-tree.

    python -m paper_2002_09049_amd.build

hipcc cross-compiles without a GPU.  Each source compiles to its own object
(in parallel, under _build/), then one link makes the shared library.
Packed-FP32 instructions are disabled (-packed-fp32-ops); the kernels never
need them.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmpq.so")
OBJ = os.path.join(ROOT, "_build", "obj")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _jobs() -> int:
    n = os.environ.get("MAX_JOBS")
    if n and n.isdigit():
        return max(1, min(int(n), 16))
    return max(1, min(len(os.sched_getaffinity(0)), 16))


def build(verbose: bool = False) -> str:
    """Always recompiles every source and relinks libmpq.so."""
    os.makedirs(OBJ, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(OBJ, os.path.basename(src)[:-4] + ".o")
        cmd = [HIPCC, *FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        p = subprocess.run(cmd, capture_output=True, text=True)
        # the host pass does not know the packed-FP32 feature: harmless
        noise = "'-packed-fp32-ops' is not a recognized feature"
        msg = "\n".join(l for l in (p.stdout + p.stderr).splitlines() if noise not in l)
        if p.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{msg}")
        if msg.strip():
            print(msg, file=sys.stderr, flush=True)
        return obj

    with ThreadPoolExecutor(_jobs()) as ex:
        objs = list(ex.map(compile_one, sources()))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    print(LIB)
    sys.exit(0)
