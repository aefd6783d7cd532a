"""Build libmoeca.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

    python -m paper_2606_15615_amd.build

Objects go to ``_build/`` at the repository root; the shared library lands
next to this file.  Decision-path and combine sources are compiled without
FMA contraction (their fp32 operations must round exactly as written).
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libmoeca.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC, "-Wall", "-Wno-unused-function",
]
SOURCES = {
    "router.hip": ["-ffp-contract=off"],
    "decide.hip": ["-ffp-contract=off"],
    "combine.hip": ["-ffp-contract=off"],
    "ffn.hip": [],
    "block.hip": ["-ffp-contract=off"],
    "noalloc.hip": [],
    "moeca.cpp": ["-ffp-contract=off"],
    "stack.cpp": [],
}


def _compile(src: str, extra: list[str]) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *COMMON, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build_library(verbose: bool = False) -> str:
    """Compile every source and link libmoeca.so; return its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        futs = {ex.submit(_compile, s, e): s for s, e in SOURCES.items()}
        objs = []
        for f in concurrent.futures.as_completed(futs):
            objs.append(f.result())
            if verbose:
                print("compiled", futs[f], flush=True)
    objs.sort()
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB, flush=True)
    return LIB


if __name__ == "__main__":
    build_library(verbose=True)
    sys.exit(0)
