"""Thin ctypes binding over libgemm_mi355x.so (argument marshalling only).

The functions named like the C entry points (``gemm_i8_i32``, ``gemm_bf16_f32``,
their column-major-B forms ``gemm_i8_i32_bt`` and ``gemm_bf16_f32_bt``, the
reduced-precision-output forms ``gemm_i8_i8``, ``gemm_i8_i16``, ``gemm_bf16_bf16``
and their ``*_bt`` forms, ``gemm_plan``,
``gemm_plan_bt``, ``gemm_force_plan``, ``gemm_force_reduce``, ``gemm_release_workspace``,
``gemm_status_string``, ``gemm_version``, the no-allocation ``gemm_bf16_f32_noalloc``
and the measurement aids ``gemm_probe_mfma`` and ``gemm_probe_read``)
take plain integers and device addresses exactly as the C ABI does.  The two
torch helpers (``mm_i8_i32``, ``mm_bf16_f32``) only read ``data_ptr()``,
strides and the current HIP stream of torch tensors and call the same entry
points; every step of the GEMM runs in the library's kernels.  There is no
fallback: if the library is missing, loading raises.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
# GEMM_MI355X_LIBRARY names another build of the same library (the sanitizer test loads a
# host-only build of the C ABI through it); there is no fallback if the file is missing.
LIB_PATH = os.environ.get("GEMM_MI355X_LIBRARY") or os.path.join(PKG, "libgemm_mi355x.so")

GEMM_OK = 0
GEMM_ERR_INVALID_VALUE = -1
GEMM_ERR_UNSUPPORTED = -2
GEMM_ERR_HIP = -3
GEMM_ERR_NO_MEMORY = -4
GEMM_ERR_SCRATCH_LIMIT = -5

GEMM_DTYPE_I8_I32 = 0
GEMM_DTYPE_BF16_F32 = 1

GEMM_KERNEL_AUTO = -1
GEMM_KERNEL_GENERIC = 0
GEMM_KERNEL_MACRO = 1
GEMM_KERNEL_SKINNY = 2
GEMM_KERNEL_DIRECT = 3
GEMM_KERNEL_RING = 4
GEMM_KERNEL_GEMV = 5

GEMM_REDUCE_SEPARATE = 0
GEMM_REDUCE_LAST_SLICE = 1
GEMM_REDUCE_ATOMIC = 2
GEMM_REDUCE_ATOMIC_FLAG = 3
# gemm_plan_info.source
GEMM_PLAN_FROM_MODEL, GEMM_PLAN_FROM_TABLE, GEMM_PLAN_FROM_NEIGHBOUR, GEMM_PLAN_FROM_FILE, GEMM_PLAN_FROM_FORCED = range(5)

EXPORTED = ("gemm_i8_i32", "gemm_bf16_f32", "gemm_i8_i32_bt", "gemm_bf16_f32_bt",
            "gemm_i8_i8", "gemm_i8_i16", "gemm_bf16_bf16", "gemm_i8_i8_bt", "gemm_i8_i16_bt",
            "gemm_bf16_bf16_bt", "gemm_plan",
            "gemm_plan_bt", "gemm_force_plan", "gemm_force_reduce", "gemm_release_workspace",
            "gemm_status_string", "gemm_version", "gemm_probe_mfma", "gemm_bf16_f32_noalloc",
            "gemm_probe_read", "gemm_load_plans", "gemm_clear_plans")


class PlanInfo(ctypes.Structure):
    _fields_ = [
        ("kernel", ctypes.c_int32), ("config", ctypes.c_int32),
        ("bm", ctypes.c_int32), ("bn", ctypes.c_int32), ("bk", ctypes.c_int32),
        ("waves", ctypes.c_int32),
        ("mfma_m", ctypes.c_int32), ("mfma_n", ctypes.c_int32), ("mfma_k", ctypes.c_int32),
        ("split_k", ctypes.c_int32), ("reduce_in_kernel", ctypes.c_int32),
        ("k_chunk", ctypes.c_int64), ("grid", ctypes.c_int64),
        ("lds_bytes", ctypes.c_int64), ("workspace_bytes", ctypes.c_int64),
        ("model_traffic_bytes", ctypes.c_double),
        ("model_t_comp_us", ctypes.c_double), ("model_t_mem_us", ctypes.c_double),
        ("source", ctypes.c_int32),
        ("name", ctypes.c_char * 48),
    ]


class ProbeInfo(ctypes.Structure):
    _fields_ = [("workgroups", ctypes.c_int64), ("threads_per_workgroup", ctypes.c_int64),
                ("ops_per_launch", ctypes.c_double), ("wall_clock_hz", ctypes.c_double)]


class GemmError(RuntimeError):
    def __init__(self, status: int):
        self.status = status
        super().__init__(gemm_status_string(status))


_lib = None


def lib() -> ctypes.CDLL:
    """Loads the built library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2512_13282_amd.build`")
        l = ctypes.CDLL(LIB_PATH)
        i64, p, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
        gemm_args = [i64, i64, i64, p, i64, p, i64, p, i64, p]
        l.gemm_i8_i32.argtypes = gemm_args
        l.gemm_i8_i32.restype = i32
        l.gemm_bf16_f32.argtypes = gemm_args
        l.gemm_bf16_f32.restype = i32
        l.gemm_i8_i32_bt.argtypes = gemm_args
        l.gemm_i8_i32_bt.restype = i32
        l.gemm_bf16_f32_bt.argtypes = gemm_args
        l.gemm_bf16_f32_bt.restype = i32
        l.gemm_bf16_f32_noalloc.argtypes = gemm_args
        l.gemm_bf16_f32_noalloc.restype = i32
        shift_args = [i64, i64, i64, p, i64, p, i64, p, i64, i32, p]
        for name in ("gemm_i8_i8", "gemm_i8_i16", "gemm_i8_i8_bt", "gemm_i8_i16_bt"):
            getattr(l, name).argtypes = shift_args
            getattr(l, name).restype = i32
        for name in ("gemm_bf16_bf16", "gemm_bf16_bf16_bt"):
            getattr(l, name).argtypes = gemm_args
            getattr(l, name).restype = i32
        plan_args = [i32, i64, i64, i64, i64, i64, i64, ctypes.c_size_t, ctypes.c_size_t,
                     ctypes.c_size_t, ctypes.POINTER(PlanInfo)]
        l.gemm_plan.argtypes = plan_args
        l.gemm_plan.restype = i32
        l.gemm_plan_bt.argtypes = plan_args
        l.gemm_plan_bt.restype = i32
        l.gemm_force_plan.argtypes = [i32, i32, i32, i32]
        l.gemm_force_plan.restype = i32
        l.gemm_force_reduce.argtypes = [i32, i32]
        l.gemm_force_reduce.restype = i32
        l.gemm_release_workspace.argtypes = []
        l.gemm_release_workspace.restype = i32
        l.gemm_load_plans.argtypes = [ctypes.c_char_p]
        l.gemm_load_plans.restype = i32
        l.gemm_clear_plans.argtypes = []
        l.gemm_clear_plans.restype = i32
        l.gemm_status_string.argtypes = [i32]
        l.gemm_status_string.restype = ctypes.c_char_p
        l.gemm_version.argtypes = []
        l.gemm_version.restype = ctypes.c_char_p
        l.gemm_probe_mfma.argtypes = [i32, i32, ctypes.c_int32, p, p, ctypes.POINTER(ProbeInfo), p]
        l.gemm_probe_mfma.restype = i32
        l.gemm_probe_read.argtypes = [p, i64, p, i64, p]
        l.gemm_probe_read.restype = i32
        _lib = l
    return _lib


# ---------------------------------------------------------------- raw C entry points
def gemm_i8_i32(M, N, K, A, lda, B, ldb, C, ldc, stream=0) -> int:
    return lib().gemm_i8_i32(M, N, K, A or None, lda, B or None, ldb, C or None, ldc, stream or None)


def gemm_bf16_f32(M, N, K, A, lda, B, ldb, C, ldc, stream=0) -> int:
    return lib().gemm_bf16_f32(M, N, K, A or None, lda, B or None, ldb, C or None, ldc, stream or None)


def gemm_bf16_f32_noalloc(M, N, K, A, lda, B, ldb, C, ldc, stream=0) -> int:
    return lib().gemm_bf16_f32_noalloc(M, N, K, A or None, lda, B or None, ldb, C or None, ldc, stream or None)


def gemm_i8_i32_bt(M, N, K, A, lda, Bt, ldbt, C, ldc, stream=0) -> int:
    return lib().gemm_i8_i32_bt(M, N, K, A or None, lda, Bt or None, ldbt, C or None, ldc, stream or None)


def gemm_bf16_f32_bt(M, N, K, A, lda, Bt, ldbt, C, ldc, stream=0) -> int:
    return lib().gemm_bf16_f32_bt(M, N, K, A or None, lda, Bt or None, ldbt, C or None, ldc, stream or None)


def gemm_i8_i8(M, N, K, A, lda, B, ldb, C, ldc, shift, stream=0) -> int:
    return lib().gemm_i8_i8(M, N, K, A or None, lda, B or None, ldb, C or None, ldc, shift, stream or None)


def gemm_i8_i16(M, N, K, A, lda, B, ldb, C, ldc, shift, stream=0) -> int:
    return lib().gemm_i8_i16(M, N, K, A or None, lda, B or None, ldb, C or None, ldc, shift, stream or None)


def gemm_bf16_bf16(M, N, K, A, lda, B, ldb, C, ldc, stream=0) -> int:
    return lib().gemm_bf16_bf16(M, N, K, A or None, lda, B or None, ldb, C or None, ldc, stream or None)


def gemm_i8_i8_bt(M, N, K, A, lda, Bt, ldbt, C, ldc, shift, stream=0) -> int:
    return lib().gemm_i8_i8_bt(M, N, K, A or None, lda, Bt or None, ldbt, C or None, ldc, shift, stream or None)


def gemm_i8_i16_bt(M, N, K, A, lda, Bt, ldbt, C, ldc, shift, stream=0) -> int:
    return lib().gemm_i8_i16_bt(M, N, K, A or None, lda, Bt or None, ldbt, C or None, ldc, shift,
                                stream or None)


def gemm_bf16_bf16_bt(M, N, K, A, lda, Bt, ldbt, C, ldc, stream=0) -> int:
    return lib().gemm_bf16_bf16_bt(M, N, K, A or None, lda, Bt or None, ldbt, C or None, ldc, stream or None)


def gemm_plan(dtype, M, N, K, lda, ldb, ldc, a_addr=0, b_addr=0, c_addr=0, trans_b=False) -> dict:
    """The selector's plan as a dict (gemm_plan, or gemm_plan_bt with trans_b=True, where
    ldb is the row stride of the N x K matrix); raises GemmError on a bad argument."""
    info = PlanInfo()
    fn = lib().gemm_plan_bt if trans_b else lib().gemm_plan
    rc = fn(dtype, M, N, K, lda, ldb, ldc, a_addr, b_addr, c_addr, ctypes.byref(info))
    if rc != GEMM_OK:
        raise GemmError(rc)
    d = {f: getattr(info, f) for f, _ in PlanInfo._fields_}
    d["name"] = info.name.decode()
    return d


def gemm_force_plan(dtype, kernel=GEMM_KERNEL_AUTO, config=-1, split_k=0) -> int:
    return lib().gemm_force_plan(dtype, kernel, config, split_k)


def gemm_force_reduce(dtype, mode=-1) -> int:
    return lib().gemm_force_reduce(dtype, mode)


def gemm_load_plans(path) -> int:
    return lib().gemm_load_plans(None if path is None else os.fsencode(path))


def gemm_clear_plans() -> int:
    return lib().gemm_clear_plans()


def gemm_release_workspace() -> int:
    return lib().gemm_release_workspace()


def gemm_status_string(status: int) -> str:
    return lib().gemm_status_string(status).decode()


def gemm_version() -> str:
    return lib().gemm_version().decode()


def gemm_probe_read(src, nbytes, sink=0, sink_elems=0, stream=0) -> int:
    return lib().gemm_probe_read(src or None, nbytes, sink or None, sink_elems, stream or None)


def gemm_probe_mfma(dtype, random_operands, iters, clocks=0, sink=0, stream=0):
    """Returns (status, info dict); with clocks == sink == 0 only the info is filled."""
    info = ProbeInfo()
    rc = lib().gemm_probe_mfma(dtype, int(bool(random_operands)), iters, clocks or None, sink or None,
                               ctypes.byref(info), stream or None)
    return rc, {f: getattr(info, f) for f, _ in ProbeInfo._fields_}


# ---------------------------------------------------------------- torch helpers
def _check(rc: int) -> None:
    if rc != GEMM_OK:
        raise GemmError(rc)


def _mm(fns, A, B, out, in_dtype, out_dtype):
    """B may be row-major (stride(1) == 1) or column-major (stride(0) == 1, e.g. W.t() of
    a contiguous N x K weight W), which selects the *_bt entry point."""
    import torch
    if A.dtype != in_dtype or B.dtype != in_dtype:
        raise TypeError(f"expected {in_dtype} operands")
    if A.dim() != 2 or B.dim() != 2 or A.shape[1] != B.shape[0]:
        raise ValueError("expected A (M x K) and B (K x N)")
    if not (A.is_cuda and B.is_cuda) or A.device != B.device:
        raise ValueError("operands must be on the same GPU")
    M, K = A.shape
    N = B.shape[1]
    if A.stride(1) != 1:
        raise ValueError("A must be row-major with unit column stride")
    trans_b = B.stride(1) != 1 and B.stride(0) == 1 and N > 1
    if not trans_b and B.stride(1) != 1 and K > 1 and N > 1:
        raise ValueError("B must be row-major or column-major")
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=A.device)
    elif out.dtype != out_dtype or tuple(out.shape) != (M, N) or out.stride(1) != 1 or out.device != A.device:
        raise ValueError("bad output tensor")
    stream = torch.cuda.current_stream(A.device).cuda_stream
    # A single-row matrix has no meaningful row stride; any value >= cols is valid.
    lda = A.stride(0) if M > 1 else max(K, 1)
    if trans_b:
        ldb = B.stride(1) if N > 1 else max(K, 1)
    else:
        ldb = B.stride(0) if K > 1 else max(N, 1)
    ldc = out.stride(0) if M > 1 else max(N, 1)
    fn = fns[1] if trans_b else fns[0]
    _check(fn(M, N, K, A.data_ptr(), lda, B.data_ptr(), ldb, out.data_ptr(), ldc, stream))
    return out


def mm_i8_i32(A, B, out=None):
    """C = A @ B for int8 torch tensors on the GPU; int32 result.  B row- or column-major."""
    import torch
    return _mm((gemm_i8_i32, gemm_i8_i32_bt), A, B, out, torch.int8, torch.int32)


def mm_bf16_f32(A, B, out=None):
    """C = A @ B for bfloat16 torch tensors on the GPU; float32 result.  B row- or column-major."""
    import torch
    return _mm((gemm_bf16_f32, gemm_bf16_f32_bt), A, B, out, torch.bfloat16, torch.float32)
