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
    fat = str(d / "fatbin.bin")
    subprocess.run([objcopy, "--dump-section", f".hip_fatbin={fat}", LIB, str(d / "stripped.so")],
                   check=True, capture_output=True)
    # One offload bundle per translation unit, back to back in the section.
    data = open(fat, "rb").read()
    magic = b"__CLANG_OFFLOAD_BUNDLE__"
    starts, i = [], data.find(magic)
    while i >= 0:
        starts.append(i)
        i = data.find(magic, i + 1)
    notes = ""
    for n, (a, b) in enumerate(zip(starts, starts[1:] + [len(data)])):
        part, co = str(d / f"bundle{n}.bin"), str(d / f"gfx950_{n}.co")
        with open(part, "wb") as f:
            f.write(data[a:b])
        subprocess.run([bundler, "--unbundle", "--type=o", f"--targets={TARGET}", f"--input={part}",
                        f"--output={co}"], check=True, capture_output=True)
        notes += subprocess.run([readelf, "--notes", co], check=True, capture_output=True, text=True).stdout
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


def _configs():
    """The tile configuration table, parsed from configs.h: one dict per row, in index order."""
    src = open(os.path.join(ROOT, "paper_2512_13282_amd", "csrc", "configs.h")).read()
    rows = re.findall(r'\{(FAM_\w+),\s*(\d+),\s*(\d+),\s*(\d+),\s*(\d+),\s*(\d+),\s*(\d+),\s*[\d.]+,\s*[\d.]+,'
                      r'\s*(\d),\s*"(\w+)"\}', src)
    keys = ("family", "bm", "bn", "wm", "wn", "occupancy", "stages", "col_major_b", "name")
    return [dict(zip(keys, (r[0], *map(int, r[1:8]), r[8]))) for r in rows]


def _config_kernels(cfg, index, kernels):
    """Kernel instances (metadata dicts) that run configuration `cfg` (both dtypes, both B layouts)."""
    f, bm, bn, wm, wn, st = cfg["family"], cfg["bm"], cfg["bn"], cfg["wm"], cfg["wn"], cfg["stages"]
    geo = rf"ELi{bm}ELi{bn}ELi{wm}ELi{wn}E"
    if f == "FAM_GENERIC":
        pat = rf"gemm_tile_kernelILi[01]{geo}Lb0E"
    elif f in ("FAM_MACRO", "FAM_SKINNY") and index not in (14, 15):
        pat = rf"gemm_vec_kernelILi[01]{geo}"
    elif index in (14, 15):
        pat = rf"gemm_stream_kernelILi[01]ELi{bm}ELi{st}E"
    elif index == 13:
        pat = r"gemm_pingpong_kernel"
    elif f == "FAM_DIRECT":
        pat = rf"gemm_lds_kernelILi[01]{geo}Li\d+ELb[01]E"
    elif f == "FAM_RING":
        pat = rf"gemm_ring_kernelILi[01]{geo}Li\d+ELb[01]ELi{st}E"
    else:
        pat = r"gemv_bt_kernel" if cfg["col_major_b"] else r"gemv_kernel"
    return {n: k for n, k in _gemm(kernels).items() if re.search(pat, n)}


def test_config_occupancy_fits_the_cu(kernels):
    """`occupancy` (workgroups resident per CU, used by the selector's wave-quantization model)
    must be what the built kernels allow: occupancy x LDS within the CU's 160 KiB, and
    occupancy x waves per SIMD x registers per wave within a SIMD's 512 registers per lane."""
    cfgs = _configs()
    assert len(cfgs) >= 41
    for i, c in enumerate(cfgs):
        ks = _config_kernels(c, i, kernels)
        assert ks, (i, c["name"])
        waves_per_simd = -(-c["wm"] * c["wn"] // 4) if c["family"] != "FAM_GEMV" else 1
        for n, k in ks.items():
            lds = int(k["group_segment_fixed_size"])
            assert c["occupancy"] * lds <= LDS_LIMIT, (c["name"], n, lds)
            regs = int(k.get("vgpr_count", 0)) + int(k.get("agpr_count", 0))
            regs = -(-regs // 8) * 8
            assert c["occupancy"] * waves_per_simd * regs <= 512, (c["name"], n, regs)
