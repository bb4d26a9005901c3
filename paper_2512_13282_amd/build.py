"""Builds libgemm_mi355x.so in-tree (gfx950 device code + host C ABI).

    python -m paper_2512_13282_amd.build          # or build() from Python

Host-only sources (the C ABI and the selector) compile with g++; the kernels
compile with hipcc for gfx950; hipcc links the shared library.  Every call
recompiles.
"""
from __future__ import annotations

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
DEVICE_SOURCES = ["gemm_kernels.hip", "mfma_probe.hip"]

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
        objs = []
        for src in HOST_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            _run(["g++", *HOST_FLAGS, "-I", os.path.join(ROOT, "include"), "-c",
                  os.path.join(CSRC, src), "-o", obj])
            objs.append(obj)
        for src in DEVICE_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            _run([HIPCC, *DEVICE_FLAGS, "-I", os.path.join(ROOT, "include"), "-c",
                  os.path.join(CSRC, src), "-o", obj])
            objs.append(obj)
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", out + ".tmp"])
        os.replace(out + ".tmp", out)
        if verbose:
            print(f"built {out}")
        return out
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


if __name__ == "__main__":
    build(verbose=True)
