"""Builds libsdb.so (the HIP library for gfx950) in-tree with hipcc.

Usage: python -m paper_2607_07632_amd.build  (or call build()).
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libsdb.so")
BUILD_DIR = os.path.join(ROOT, "_build")

# the fused pass's instances are spread over several files so they compile in parallel
SOURCES = ["sdb_api.cpp", "sdb_kernels.hip", "sdb_fused_vec.hip", "sdb_fused_rows.hip", "sdb_fused_eager.hip",
           "sdb_fused_big.hip", "sdb_fused_unroll.hip", "sdb_fused_unroll_big.hip"]

COMMON = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-fvisibility=hidden",
    "-Wall",
    "-Wno-unused-function",
    # no packed fp32 instructions anywhere (the path is integer-only anyway)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE,
    "-I", CSRC,
]


def _hipcc() -> str:
    h = os.environ.get("HIPCC") or shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(h):
        raise RuntimeError(f"hipcc not found ({h})")
    return h


def _rocm(hipcc: str) -> str:
    return os.environ.get("ROCM_PATH") or os.path.dirname(os.path.dirname(os.path.realpath(hipcc)))


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


def build(verbose: bool = False, extra_flags: list[str] | None = None) -> str:
    """Compiles every source for gfx950 and links libsdb.so next to this file."""
    hipcc = _hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    flags = COMMON + list(extra_flags or [])
    objs = []
    jobs = []
    for src in SOURCES:
        obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
        lang = (["-x", "hip"] if src.endswith(".hip")
                else ["-x", "c++", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(_rocm(hipcc), "include")])
        jobs.append([hipcc] + flags + lang + ["-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    with ThreadPoolExecutor(max_workers=len(jobs)) as ex:
        list(ex.map(lambda c: _run(c, verbose), jobs))
    fd, tmp = tempfile.mkstemp(prefix="libsdb.", suffix=".so.tmp", dir=PKG)
    os.close(fd)
    try:
        _run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs, verbose)
        os.replace(tmp, LIB)
    finally:
        if os.path.exists(tmp):
            os.unlink(tmp)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
