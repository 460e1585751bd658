"""Builds libvsr.so (the HIP library behind include/vsr.h) for gfx950.

Run as ``python -m paper_2601_01513_amd.build``. Objects go to ``_build/``
at the repository root; the library lands next to this file.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libvsr.so")

SOURCES = ["vsr.cpp", "kernels_misc.hip", "kernels_simple.hip", "kernels_gemm.hip",
           "kernels_attn.hip", "kernels_retrieval.hip", "kernels_skinny.hip"]

# -packed-fp32-ops: keep hipcc from emitting packed fp32 VALU instructions.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-x", "hip",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", INCLUDE, "-I", CSRC]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found")
    return path


def _quiet(stderr: str) -> str:
    # The host pass does not know the gfx950 feature flag above; drop that note.
    return "\n".join(l for l in stderr.splitlines()
                     if "packed-fp32-ops" not in l)


def _compile(src: str, extra) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [hipcc(), *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{_quiet(r.stderr)}")
    msg = _quiet(r.stderr).strip()
    if msg:
        print(msg, file=sys.stderr)
    return obj


def build(extra=(), jobs: int = 8) -> str:
    """Compiles every source and links libvsr.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, list(extra)), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
