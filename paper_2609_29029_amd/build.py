"""Build librift.so (the HIP kernels and the C ABI) for gfx950 with hipcc, and
libriftcalib.so, a measurement aid for the benchmark (the MFMA throughput
ceiling), which nothing on the Rift path loads.

Usage: python -m paper_2609_29029_amd.build   (or build() from Python).
Every call recompiles; objects go to _build/ next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "librift.so")
CALIB_OUT = os.path.join(HERE, "libriftcalib.so")
BUILD = os.path.join(HERE, "_build")

SOURCES = ["score.hip", "knn.hip", "select.hip", "merge.hip", "compact.hip", "prefill_misc.hip", "gemm_bf16.hip",
           "gemm_skinny.hip", "attention.hip", "decode.hip", "debug.hip", "capi.hip"]
CALIB_SOURCES = ["calib/mfma_ceiling.hip"]

ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-Wall",
         "-Wno-unused-function", "-Wno-pass-failed", "-fvisibility=hidden",
         # no packed fp32 instructions in any kernel
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0].replace("/", "_") + ".o")
    cmd = [hipcc(), *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def _link(objs, out: str) -> None:
    tmp = out + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = SOURCES + CALIB_SOURCES
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    _link(objs[:len(SOURCES)], OUT)
    _link(objs[len(SOURCES):], CALIB_OUT)
    if verbose:
        print(f"built {OUT} and {CALIB_OUT}")
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
