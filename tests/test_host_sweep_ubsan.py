"""CPU-only: the library's host code (argument checks, screen and split planners, workspace sizers and
every launcher's grid arithmetic) compiled for the host alone under -fsanitize=undefined and driven over
degenerate shapes by tests/host_sweep.cpp.  An integer division by zero, a signed overflow or an
out-of-range shift in any of it aborts the driver.  No GPU is used: the device pointers are fake and
every launch fails for lack of a device after its host-side arithmetic has run."""
import concurrent.futures as cf
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2412_09282_amd", "csrc")
HIPCC = "/opt/rocm/bin/hipcc"
SAN = ["-Xarch_host", "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=undefined"]
FLAGS = ["--offload-host-only", "-O1", "-g", "-std=c++17", "-I", os.path.join(ROOT, "include"), "-I", CSRC] + SAN


def _run(cmd, cwd):
    r = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r.stdout


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_host_code_under_ubsan():
    srcs = sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))
    tmp = tempfile.mkdtemp(prefix="crvq_ubsan_")
    try:
        jobs = [[HIPCC] + FLAGS + ["-c", os.path.join(CSRC, f), "-o", f.replace(".hip", ".o")] for f in srcs]
        jobs.append([HIPCC] + FLAGS + ["-x", "hip", "-c", os.path.join(ROOT, "tests", "host_sweep.cpp"), "-o",
                                        "sweep.o"])
        with cf.ThreadPoolExecutor(max_workers=4) as ex:
            list(ex.map(lambda c: _run(c, tmp), jobs))
        objs = sorted(f for f in os.listdir(tmp) if f.endswith(".o"))
        # host-only objects name the device images a full build would embed; empty stand-ins let the
        # driver link (no kernel is ever loaded without a device)
        und = _run(["nm", "-u"] + objs, tmp)
        syms = sorted({ln.split()[-1] for ln in und.splitlines() if "__hip_fatbin_" in ln})
        with open(os.path.join(tmp, "fatbin_stub.c"), "w") as f:
            for s in syms:
                f.write(f"char {s}[4096] __attribute__((aligned(4096))) = {{0}};\n")
        _run(["gcc", "-c", "fatbin_stub.c", "-o", "fatbin_stub.o"], tmp)
        _run([HIPCC, "-Xarch_host", "-fsanitize=undefined", "-o", "sweep"] + objs + ["fatbin_stub.o",
                                                                          "-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx",
                                                                          "-Wl,-rpath,/opt/rocm/lib"], tmp)
        r = subprocess.run(["./sweep"], cwd=tmp, capture_output=True, text=True, timeout=300,
                           env=dict(os.environ, UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1"))
        assert r.returncode == 0, f"host sweep failed:\n{r.stdout}\n{r.stderr}"
        assert "host sweep ok" in r.stdout and "runtime error" not in r.stderr, r.stdout + r.stderr
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
