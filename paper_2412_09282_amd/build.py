"""Build libcrvq.so for gfx950 with hipcc (in-tree, no JIT cache).

    python -m paper_2412_09282_amd.build        # compile every translation unit and link

Each kernel file compiles on its own; the screen kernels additionally get
-fno-honor-nans (lets min/med3 run without NaN canonicalisation; inputs must be
finite) and the VGPR form of MFMA (results land in VGPRs, no accumulator copies).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libcrvq.so")
ARCH = "gfx950"

SOURCES = {
    "api.hip": [],
    "k_screen.hip": ["-fno-honor-nans", "-mllvm", "-amdgpu-mfma-vgpr-form=1"],
    "k_kmeans.hip": [],
    "k_colreduce.hip": [],
    "k_reorder.hip": [],
    "k_dequant.hip": [],
    "k_gemv.hip": [],
    "k_refine.hip": [],
    "k_hinv.hip": [],
}

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    # packed fp32 VALU forms are disabled for every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-pass-failed", "-I", INCLUDE, "-I", CSRC,
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return "hipcc"


def _compile(src: str, extra) -> str:
    obj = os.path.join(BUILD_DIR, src.replace(".hip", ".o"))
    cmd = [hipcc()] + COMMON + list(extra) + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = True) -> str:
    """Compile all translation units for gfx950 and link libcrvq.so; returns its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        futs = {ex.submit(_compile, s, e): s for s, e in SOURCES.items()}
        objs = []
        for f in cf.as_completed(futs):
            objs.append(f.result())
            if verbose:
                print(f"[crvq build] compiled {futs[f]}", flush=True)
    tmp = LIB + f".tmp{os.getpid()}"
    # roctx: the profiler ranges around the entry points
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + sorted(objs) + [
        "-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-Wl,-rpath,/opt/rocm/lib"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"[crvq build] linked {LIB}", flush=True)
    return LIB


def exported_symbols() -> list:
    """Names of the C functions declared in include/crvq.h."""
    import re
    text = open(os.path.join(INCLUDE, "crvq.h")).read()
    return sorted(set(re.findall(r"\b(crvq_[a-z0-9_]+)\s*\(", text)))


if __name__ == "__main__":
    build()
    sys.exit(0)
