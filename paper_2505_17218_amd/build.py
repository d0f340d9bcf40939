"""Build libdash.so (the HIP kernels and the C ABI of include/dash.h) for gfx950.

Usage: python -m paper_2505_17218_amd.build   (or __graft_entry__.build()).
Compiles every library source in csrc/ with hipcc into one shared library next to
this file, the native benchmark (csrc/native_bench.hip, a C-ABI client that needs
no Python) into dash_native_bench, and the projection-GEMM micro-benchmark
(csrc/gemm_bench.hip) into dash_gemm_bench beside it.  The sampler and advantage
kernels are built with -ffp-contract=off: their float32 arithmetic is part of a
bit-exact contract.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libdash.so")
NATIVE_BENCH = os.path.join(HERE, "dash_native_bench")
GEMM_BENCH = os.path.join(HERE, "dash_gemm_bench")
BUILD = os.path.join(ROOT, "_build")

SOURCES = ["runtime.hip", "elementwise.hip", "gemm.hip", "attention.hip", "sampler.hip", "advantage.hip"]
EXACT = {"sampler.hip", "advantage.hip"}

COMMON = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def hipcc() -> str:
    return shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src.replace(".hip", ".o"))
    flags = list(COMMON)
    if src in EXACT:
        flags += ["-ffp-contract=off"]
    else:
        flags += ["-ffp-contract=fast"]
    cmd = [hipcc(), *flags, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    tmp = NATIVE_BENCH + ".tmp"
    cmd = [hipcc(), *COMMON, "-ffp-contract=fast", os.path.join(CSRC, "native_bench.hip"), "-o", tmp,
           "-L", HERE, "-ldash", "-Wl,-rpath,$ORIGIN"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"native benchmark build failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, NATIVE_BENCH)
    tmp = GEMM_BENCH + ".tmp"
    cmd = [hipcc(), *COMMON, "-ffp-contract=fast", os.path.join(CSRC, "gemm_bench.hip"), "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"GEMM benchmark build failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, GEMM_BENCH)
    if verbose:
        print(f"built {LIB}, {NATIVE_BENCH} and {GEMM_BENCH}", file=sys.stderr)
    return LIB


if __name__ == "__main__":
    build()
