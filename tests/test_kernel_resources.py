"""Resource use of the built gfx950 kernels, read from the library's own code object.

A GEMM kernel whose accumulator tile does not stay in registers runs an order of
magnitude slower (a 256 x 256 int8 tile over four waves once went to 1152 bytes of
scratch per lane when its epilogue loops stopped unrolling, and took 10 ms instead
of 0.5 ms at 8192^3), yet computes the same result, so parity tests cannot see it.
This test reads the AMDGPU metadata notes of the gfx950 code object inside the
built library and bounds what each GEMM kernel uses.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2512_13282_amd", "libgemm_mi355x.so")
LLVM = "/opt/rocm/llvm/bin"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"
LDS_LIMIT = 160 * 1024                 # bytes of LDS one workgroup may use on gfx950
# Bytes of scratch per lane: room for some spilled registers (the 4-wave 256 x 256 bf16
# ring kernels spill about 60 in their epilogue), far below an accumulator tile (1 KiB+).
SCRATCH_LIMIT = 256


def _tool(name):
    p = os.path.join(LLVM, name)
    return p if os.path.exists(p) else shutil.which(name)


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    tools = [_tool(t) for t in ("llvm-objcopy", "clang-offload-bundler", "llvm-readelf")]
    if not os.path.exists(LIB) or not all(tools):
        pytest.skip("library not built or LLVM tools missing")
    objcopy, bundler, readelf = tools
    d = tmp_path_factory.mktemp("codeobj")
    fat, co = str(d / "fatbin.bin"), str(d / "gfx950.co")
    subprocess.run([objcopy, "--dump-section", f".hip_fatbin={fat}", LIB, str(d / "stripped.so")],
                   check=True, capture_output=True)
    subprocess.run([bundler, "--unbundle", "--type=o", f"--targets={TARGET}", f"--input={fat}",
                    f"--output={co}"], check=True, capture_output=True)
    notes = subprocess.run([readelf, "--notes", co], check=True, capture_output=True, text=True).stdout
    out, cur = {}, None
    for line in notes.splitlines():
        m = re.match(r"\s*(?:- )?\.(\w+):\s+(\S+)", line)
        if not m:
            continue
        key, val = m.groups()
        if line.lstrip().startswith("- ."):
            cur = {}
        if cur is None:
            continue
        cur[key] = val
        if key == "name" and not val.endswith(".kd"):
            out[val] = cur
    return out


def _gemm(kernels):
    """The GEMM and GEMV kernels (namespace gemm), without the split-K helpers."""
    return {n: k for n, k in kernels.items()
            if n.startswith("_ZN4gemm") and ("gemm_" in n or "gemv_" in n)}


def test_every_gemm_kernel_present(kernels):
    names = _gemm(kernels)
    for fam in ("gemm_lds_kernel", "gemm_ring_kernel", "gemm_tile_kernel", "gemm_vec_kernel",
                "gemm_stream_kernel", "gemv_kernel", "gemv_bt_kernel"):
        assert any(fam in n for n in names), fam


def test_gemm_kernels_keep_accumulators_in_registers(kernels):
    over = {n: int(k["private_segment_fixed_size"]) for n, k in _gemm(kernels).items()
            if int(k.get("private_segment_fixed_size", 0)) > SCRATCH_LIMIT}
    assert not over, f"kernels using more than {SCRATCH_LIMIT} B of scratch per lane: {over}"


def test_8192_plan_kernels_use_no_scratch(kernels):
    # direct_256x256_w8t, the plan of every 8192^3 case, and its ring counterpart.
    for pat in (r"gemm_lds_kernelILi[01]ELi256ELi256ELi4ELi2ELi2ELb[01]E",
                r"gemm_ring_kernelILi[01]ELi256ELi256ELi4ELi2ELi2ELb[01]ELi[45]E"):
        hits = {n: k for n, k in _gemm(kernels).items() if re.search(pat, n)}
        assert len(hits) >= 4, pat
        for n, k in hits.items():
            assert int(k["private_segment_fixed_size"]) == 0, n
            assert int(k.get("vgpr_spill_count", 0)) == 0, n


def test_lds_within_limit(kernels):
    for n, k in _gemm(kernels).items():
        assert int(k["group_segment_fixed_size"]) <= LDS_LIMIT, n
