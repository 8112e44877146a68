"""Build libbk.so (the HIP kernels and the C ABI of include/bk.h) for gfx950.

    python paper_2210_00038_amd/build.py [--ceiling]

Every source is compiled by hipcc into an object in ``_build/`` (in parallel),
then linked into ``paper_2210_00038_amd/libbk.so``.  Packed-fp32 instruction
selection is switched off for all device code.  ``--ceiling`` also builds
``_build/gemm_loop``, the standalone microbenchmark of the clipped-gradient
GEMM's inner loop (csrc/ceiling/gemm_loop.hip).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libbk.so")

SOURCES = ["api.cpp", "ghost_norm.hip", "agemm.hip", "clip_noise.hip", "embed_grad.hip", "wsum.hip", "conv_prep.hip", "affine.hip", "noalloc.hip", "embed_join.hip", "plan.cpp"]

ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", f"-I{INCLUDE}", f"-I{CSRC}"]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found: the HIP toolchain (ROCm) is required to build libbk")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [hipcc(), *FLAGS, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking libbk.so failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


def build_ceiling(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    exe = os.path.join(BUILD, "gemm_loop")
    flags = [f for f in FLAGS if f != "-fPIC"]
    cmd = [hipcc(), *flags, "-x", "hip", os.path.join(CSRC, "ceiling", "gemm_loop.hip"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling the GEMM-loop microbenchmark failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    if verbose:
        print(f"built {exe}")
    return exe


if __name__ == "__main__":
    build(verbose=True)
    if "--ceiling" in sys.argv[1:]:
        build_ceiling(verbose=True)
    sys.exit(0)
