"""The CPU-side code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The oracle (oracle/oracle_gemm.c) is rebuilt with -fsanitize=address,undefined and
  every oracle pin runs against that build.
* The C ABI and the selector (csrc/gemm_api.cpp, csrc/selector.cpp) are rebuilt as a
  host-only library (tests/sanitize_stub.cpp stands in for the device side, which these
  tests never reach) with the same sanitizers, and the CPU ABI, selector and plan-file
  tests run against it.

Each run is a child Python process with the ASan runtime preloaded; any sanitizer report
aborts the child and fails the test."""
import os
import subprocess
import sys

import pytest

from oracle import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2512_13282_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]


def _runtime():
    p = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not p or not os.path.exists(p):
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    return p


def _env(extra=None):
    env = dict(os.environ)
    env["LD_PRELOAD"] = _runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env.update(extra or {})
    return env


_PINS = r"""
import sys
sys.path[:0] = [{root!r}, {here!r}]
from oracle import oracle
import oracle_pins
o = oracle.Oracle({lib!r})
for p in oracle_pins.PINS:
    p(o)
print("pins ok", len(oracle_pins.PINS))
"""


def test_oracle_pins_under_sanitizers(tmp_path):
    lib = oracle.build(out=str(tmp_path / "liboracle_san.so"), extra_flags=SAN)
    r = subprocess.run([sys.executable, "-c", _PINS.format(root=ROOT, here=HERE, lib=lib)], env=_env(),
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0 and "pins ok" in r.stdout, r.stdout[-2000:] + r.stderr[-4000:]


def test_c_abi_and_selector_under_sanitizers(tmp_path):
    out = str(tmp_path / "libgemm_host_san.so")
    cmd = ["g++", "-std=c++17", "-O1", "-shared", "-fPIC", *SAN, "-I", os.path.join(ROOT, "include"),
           os.path.join(CSRC, "gemm_api.cpp"), os.path.join(CSRC, "selector.cpp"),
           os.path.join(HERE, "sanitize_stub.cpp"), "-o", out]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(HERE, "test_abi_cpu.py"), os.path.join(HERE, "test_selector.py"),
                        os.path.join(HERE, "test_plan_file.py")],
                       env=_env({"GEMM_MI355X_LIBRARY": out}), capture_output=True, text=True, timeout=600,
                       cwd=ROOT)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert " passed" in r.stdout
