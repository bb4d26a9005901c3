"""The C-ABI library on a machine without a GPU: it loads, exports every declared
entry point, rejects bad arguments before any HIP call, and plans on the host."""
import os
import re

import pytest

from paper_2512_13282_amd import binding as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gemm_mi355x.h")

I8, BF = b.GEMM_DTYPE_I8_I32, b.GEMM_DTYPE_BF16_F32
FAKE_A, FAKE_B, FAKE_C = 0x10000000, 0x20000000, 0x40000000   # never dereferenced


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(gemm_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(b.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = b.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings_and_version():
    for rc in (b.GEMM_OK, b.GEMM_ERR_INVALID_VALUE, b.GEMM_ERR_UNSUPPORTED, b.GEMM_ERR_HIP,
               b.GEMM_ERR_NO_MEMORY, b.GEMM_ERR_SCRATCH_LIMIT):
        assert b.gemm_status_string(rc).startswith("GEMM_")
    assert "unknown" in b.gemm_status_string(12345)
    assert "gfx950" in b.gemm_version()


@pytest.mark.parametrize("fn", [b.gemm_i8_i32, b.gemm_bf16_f32, b.gemm_bf16_f32_noalloc])
@pytest.mark.parametrize("args", [
    (-1, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4),     # negative M
    (4, -1, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4),     # negative N
    (4, 4, -1, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4),     # negative K
    (4, 4, 8, FAKE_A, 7, FAKE_B, 4, FAKE_C, 4),      # lda < K
    (4, 8, 4, FAKE_A, 4, FAKE_B, 7, FAKE_C, 8),      # ldb < N
    (4, 8, 4, FAKE_A, 4, FAKE_B, 8, FAKE_C, 7),      # ldc < N
    (4, 4, 4, 0, 4, FAKE_B, 4, FAKE_C, 4),           # null A
    (4, 4, 4, FAKE_A, 4, 0, 4, FAKE_C, 4),           # null B
    (4, 4, 4, FAKE_A, 4, FAKE_B, 4, 0, 4),           # null C
    (4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_A + 8, 4),  # C overlaps A
    (4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_B, 4),      # C aliases B
    (4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C + 2, 4),  # C not 4-byte aligned
    (4, 4, 4, FAKE_A, 1 << 62, FAKE_B, 4, FAKE_C, 4),  # stride overflow
])
def test_invalid_arguments_rejected_before_hip(fn, args):
    assert fn(*args, 0) == b.GEMM_ERR_INVALID_VALUE


def test_bf16_pointer_alignment():
    assert b.gemm_bf16_f32(4, 4, 4, FAKE_A + 1, 4, FAKE_B, 4, FAKE_C, 4, 0) == b.GEMM_ERR_INVALID_VALUE


@pytest.mark.parametrize("fn", [b.gemm_i8_i32, b.gemm_bf16_f32, b.gemm_bf16_f32_noalloc])
def test_empty_output_is_a_noop(fn):
    # M == 0 or N == 0: nothing to write, success without touching the GPU; pointers of
    # empty operands may be null, those of non-empty ones may not
    assert fn(0, 5, 7, 0, 7, FAKE_B, 5, 0, 5, 0) == b.GEMM_OK
    assert fn(3, 0, 7, FAKE_A, 7, 0, 1, 0, 1, 0) == b.GEMM_OK
    assert fn(0, 0, 0, 0, 1, 0, 1, 0, 1, 0) == b.GEMM_OK
    assert fn(0, 5, 7, 0, 7, 0, 5, 0, 5, 0) == b.GEMM_ERR_INVALID_VALUE   # B is 7 x 5, not empty


def test_force_plan_validation():
    assert b.gemm_force_plan(7, -1, -1, 0) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_force_plan(I8, 9, -1, 0) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_force_plan(I8, -1, 999, 0) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_force_plan(I8, -1, -1, -3) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_force_plan(I8, b.GEMM_KERNEL_GENERIC, 2, 0) == b.GEMM_ERR_INVALID_VALUE  # family mismatch
    assert b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, -1, 0) == b.GEMM_OK


def test_force_reduce_validation():
    assert b.gemm_force_reduce(7, 0) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_force_reduce(I8, 4) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_force_reduce(I8, -2) == b.GEMM_ERR_INVALID_VALUE
    for mode in (b.GEMM_REDUCE_SEPARATE, b.GEMM_REDUCE_LAST_SLICE, b.GEMM_REDUCE_ATOMIC,
                 b.GEMM_REDUCE_ATOMIC_FLAG, -1):
        assert b.gemm_force_reduce(I8, mode) == b.GEMM_OK


def test_plan_invalid_arguments():
    with pytest.raises(b.GemmError):
        b.gemm_plan(I8, 4, 4, 4, 3, 4, 4, FAKE_A, FAKE_B, FAKE_C)
    with pytest.raises(b.GemmError):
        b.gemm_plan(5, 4, 4, 4, 4, 4, 4, FAKE_A, FAKE_B, FAKE_C)


@pytest.mark.parametrize("fn", [b.gemm_i8_i32_bt, b.gemm_bf16_f32_bt])
@pytest.mark.parametrize("args", [
    (-1, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4),     # negative M
    (4, 8, 16, FAKE_A, 16, FAKE_B, 15, FAKE_C, 8),   # ldbt < K (Bt is N x K)
    (4, 4, 4, FAKE_A, 4, 0, 4, FAKE_C, 4),           # null Bt
    (4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_B + 4, 4),  # C overlaps Bt
    (4, 4, 4, FAKE_A, 4, FAKE_B, 1 << 62, FAKE_C, 4),  # stride overflow
])
def test_bt_invalid_arguments_rejected_before_hip(fn, args):
    assert fn(*args, 0) == b.GEMM_ERR_INVALID_VALUE


def test_bt_strides_follow_the_n_by_k_layout():
    # Bt is N x K: a row stride >= K is valid even when it is < N, which the row-major
    # entry point (rows of N) rejects
    p = b.gemm_plan(I8, 64, 512, 128, 128, 128, 512, FAKE_A, FAKE_B, FAKE_C, trans_b=True)
    assert p["split_k"] >= 1
    with pytest.raises(b.GemmError):
        b.gemm_plan(I8, 64, 512, 128, 128, 128, 512, FAKE_A, FAKE_B, FAKE_C)
    assert b.gemm_i8_i32_bt(0, 5, 7, 0, 7, FAKE_B, 7, 0, 5, 0) == b.GEMM_OK


@pytest.mark.parametrize("fn", [b.gemm_i8_i8, b.gemm_i8_i16, b.gemm_i8_i8_bt, b.gemm_i8_i16_bt])
def test_requant_shift_range(fn):
    for shift in (-1, 32, 1000):
        assert fn(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 4, shift, 0) == b.GEMM_ERR_INVALID_VALUE
    assert fn(0, 4, 4, 0, 4, FAKE_B, 4, 0, 4, 31, 0) == b.GEMM_OK          # empty: no-op


def test_reduced_output_alignment_and_overlap():
    # int16 / bf16 outputs need 2-byte alignment, int8 outputs none
    assert b.gemm_i8_i16(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C + 1, 4, 0, 0) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_bf16_bf16(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C + 1, 4, 0) == b.GEMM_ERR_INVALID_VALUE
    # a 4 x 4 int8 C starting inside A overlaps it
    assert b.gemm_i8_i8(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_A + 15, 4, 0, 0) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_i8_i16(4, 4, 4, FAKE_A + 8, 4, FAKE_B, 4, FAKE_A, 4, 0, 0) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_i8_i8(4, 4, 4, FAKE_A, 4, FAKE_B, 4, FAKE_C, 3, 0, 0) == b.GEMM_ERR_INVALID_VALUE  # ldc < N
    assert b.gemm_bf16_bf16_bt(4, 8, 16, FAKE_A, 16, FAKE_B, 15, FAKE_C, 8, 0) == b.GEMM_ERR_INVALID_VALUE
