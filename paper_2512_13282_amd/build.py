"""Builds libgemm_mi355x.so in-tree (gfx950 device code + host C ABI).

    python -m paper_2512_13282_amd.build          # or build() from Python

Host-only sources (the C ABI and the selector) compile with g++; the kernel
translation units (one per kernel family, see csrc/families.h) compile with
hipcc for gfx950, in parallel; hipcc links the shared library.  Every call
recompiles.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libgemm_mi355x.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HOST_SOURCES = ["gemm_api.cpp", "selector.cpp"]
DEVICE_SOURCES = sorted(os.path.basename(p) for p in glob.glob(os.path.join(CSRC, "*.hip")))

# Packed-fp32 instructions are disabled for all device code (the hipcc host
# pass warns that it does not know the feature; that warning is harmless).
DEVICE_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-Wno-unused-command-line-argument"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra"]


def _run(cmd: list[str]) -> None:
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd)}")


def build(out: str = LIB, verbose: bool = False) -> str:
    tmp = tempfile.mkdtemp(prefix="gemm_build_")
    try:
        jobs = []
        for src in HOST_SOURCES:
            jobs.append(["g++", *HOST_FLAGS, "-I", os.path.join(ROOT, "include"), "-c",
                         os.path.join(CSRC, src), "-o", os.path.join(tmp, src + ".o")])
        for src in DEVICE_SOURCES:
            jobs.append([HIPCC, *DEVICE_FLAGS, "-I", os.path.join(ROOT, "include"), "-c",
                         os.path.join(CSRC, src), "-o", os.path.join(tmp, src + ".o")])
        objs = [j[-1] for j in jobs]
        # The slowest translation units (the ring and direct families) first, one compiler per core.
        weight = lambda j: next((i for i, k in enumerate(("ring", "direct", "tile")) if k in j[-3]), 3)
        jobs.sort(key=weight)
        workers = max(1, min(len(jobs), os.cpu_count() or 1, 16))
        with cf.ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(_run, jobs))
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", out + ".tmp"])
        os.replace(out + ".tmp", out)
        if verbose:
            print(f"built {out}")
        return out
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


if __name__ == "__main__":
    build(verbose=True)
