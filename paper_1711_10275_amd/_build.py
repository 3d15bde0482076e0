"""Compile the HIP sources of libsscn.so for gfx950 (hipcc, in-tree).

Each translation unit is compiled to an object under ``_build/`` in
parallel, then linked into ``paper_1711_10275_amd/libsscn.so`` (csrc/) and
``libsscn_measure.so`` (measure/: the benchmark's measured ceilings).  The library
is always rebuilt (a stale .so must never survive a source change); the
final rename is atomic so a reader never sees a half-written file.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libsscn.so")
MEASURE = os.path.join(PKG, "measure")
MEASURE_LIB = os.path.join(PKG, "libsscn_measure.so")

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 instructions are kept out of all device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # fp32 atomic adds in wgrad map to the hardware instruction
    "-munsafe-fp-atomics",
    # MFMA results go straight to VGPRs: no accumulator-register reads in the
    # inner loops (VALU work beyond ~2 instructions per fp32 MFMA is not
    # hidden behind the matrix unit)
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wall", "-Wno-unused-function",
    "-I", INCLUDE, "-I", CSRC,
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def _link(objs, lib):
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Build libsscn.so (the layers) and libsscn_measure.so (the measured
    ceilings that the benchmark reports beside the datasheet peaks)."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    msrcs = sorted(glob.glob(os.path.join(MEASURE, "*.hip")))
    workers = min(len(srcs) + len(msrcs), int(os.environ.get("MAX_JOBS", os.cpu_count() or 4)), 16)
    with cf.ThreadPoolExecutor(max_workers=max(1, workers)) as ex:
        objs = list(ex.map(_compile, srcs + msrcs))
    _link(objs[:len(srcs)], LIB)
    _link(objs[len(srcs):], MEASURE_LIB)
    if verbose:
        print(f"built {LIB} and {MEASURE_LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
