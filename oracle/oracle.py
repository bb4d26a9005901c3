"""ctypes front end of the CPU GEMM oracle (``oracle_gemm.c``).

TEST INFRASTRUCTURE ONLY: the test suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` are the only callers.  Nothing here imports or
calls the GPU package; the two share no code.

The oracle computes ``C = A @ B`` for row-major A (M x K) and B (K x N) -- the
GEMM problem of the paper, Sec. 4.1 (Multi-Level Tiling Method), with the
row-major layouts of Sec. 4.2.2 (Memory Tile Design):

* int8 -> int32: exact int64 accumulation, then an int32 range check;
* bf16 -> fp64 : operands widened exactly, exact products, fp64 sum with k
  ascending.

Every function takes numpy arrays (2-D, row stride free, unit column stride).

``requant_i32`` and ``round_bf16`` turn exact results into the reduced output
precisions the paper also reports (int8 -> int8 / int16, bf16 -> bf16; Sec. 5.1,
Sec. 5.2.3), by the rounding rules stated in ``oracle_gemm.c`` (the paper gives
none).

The ``*_bt`` forms take B stored column-major, i.e. as its transpose Bt (N x K),
the layout the paper prefers for B (Sec. 4.3).  They form B = Bt^T with a plain
transposing copy and call the row-major routine: the same products summed in
the same k order.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "oracle_gemm.c")
LIB = os.path.join(_HERE, "liboracle_gemm.so")

# -O2, no -ffast-math: the fp64 sum over k must not be reassociated.
CFLAGS = ["-O2", "-fPIC", "-shared", "-pthread", "-std=c11", "-fno-fast-math"]


def build(src: str = SRC, out: str = LIB, extra_flags: list[str] | None = None) -> str:
    """Compile the oracle with gcc into ``out`` (always recompiles)."""
    cmd = ["gcc", *CFLAGS, *(extra_flags or []), src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


class Oracle:
    """Loaded oracle library.  ``Oracle(path)`` loads a specific build."""

    def __init__(self, path: str = LIB):
        if path == LIB and not os.path.exists(path):
            build()
        self.path = path
        lib = ctypes.CDLL(path)
        i64, p = ctypes.c_int64, ctypes.c_void_p
        lib.oracle_gemm_i8_i32.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64,
                                           ctypes.c_int, ctypes.POINTER(i64)]
        lib.oracle_gemm_i8_i32.restype = ctypes.c_int
        lib.oracle_gemm_i8_i64.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64, ctypes.c_int]
        lib.oracle_gemm_i8_i64.restype = ctypes.c_int
        lib.oracle_gemm_bf16_f64.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64, ctypes.c_int]
        lib.oracle_gemm_bf16_f64.restype = ctypes.c_int
        lib.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
        lib.oracle_bf16_to_double.restype = ctypes.c_double
        lib.oracle_freivalds_i8_i32.argtypes = [i64, i64, i64, p, i64, p, i64, p, i64,
                                                ctypes.c_int, ctypes.c_uint64]
        lib.oracle_freivalds_i8_i32.restype = i64
        lib.oracle_requant_i32.argtypes = [p, i64, ctypes.c_int, ctypes.c_int, p]
        lib.oracle_requant_i32.restype = ctypes.c_int
        lib.oracle_round_bf16.argtypes = [p, i64, p]
        lib.oracle_round_bf16.restype = ctypes.c_int
        lib.oracle_bf16_from_double.argtypes = [ctypes.c_double]
        lib.oracle_bf16_from_double.restype = ctypes.c_uint16
        self.lib = lib

    # -- helpers -----------------------------------------------------------
    @staticmethod
    def _ld(x: np.ndarray) -> int:
        assert x.ndim == 2 and x.strides[1] == x.itemsize, "row-major, unit column stride"
        return x.strides[0] // x.itemsize

    @staticmethod
    def threads(n: int | None) -> int:
        return n if n else len(os.sched_getaffinity(0))

    # -- GEMMs ---------------------------------------------------------------
    @staticmethod
    def _out(M: int, N: int, dtype, ldc_pad: int):
        """Output buffer with row stride N + ldc_pad; returns (view, buffer, ldc)."""
        ldc = N + ldc_pad
        buf = np.full((M, max(ldc, 1)), 77, dtype=dtype)
        return buf[:, :N], buf, max(ldc, 1)

    def gemm_i8_i32(self, A: np.ndarray, B: np.ndarray, nthreads: int | None = None,
                    ldc_pad: int = 0):
        """Returns (C int32 M x N, overflow_count)."""
        assert A.dtype == np.int8 and B.dtype == np.int8 and A.shape[1] == B.shape[0]
        M, K = A.shape
        N = B.shape[1]
        C, buf, ldc = self._out(M, N, np.int32, ldc_pad)
        ovf = ctypes.c_int64(0)
        rc = self.lib.oracle_gemm_i8_i32(M, N, K, A.ctypes.data, self._ld(A) if M and K else max(K, 1),
                                         B.ctypes.data, self._ld(B) if K and N else max(N, 1),
                                         buf.ctypes.data, ldc, self.threads(nthreads),
                                         ctypes.byref(ovf))
        if rc != 0:
            raise RuntimeError(f"oracle_gemm_i8_i32 failed ({rc})")
        return C, int(ovf.value)

    def gemm_i8_i64(self, A: np.ndarray, B: np.ndarray, nthreads: int | None = None,
                    ldc_pad: int = 0) -> np.ndarray:
        assert A.dtype == np.int8 and B.dtype == np.int8 and A.shape[1] == B.shape[0]
        M, K = A.shape
        N = B.shape[1]
        C, buf, ldc = self._out(M, N, np.int64, ldc_pad)
        rc = self.lib.oracle_gemm_i8_i64(M, N, K, A.ctypes.data, self._ld(A) if M and K else max(K, 1),
                                         B.ctypes.data, self._ld(B) if K and N else max(N, 1),
                                         buf.ctypes.data, ldc, self.threads(nthreads))
        if rc != 0:
            raise RuntimeError(f"oracle_gemm_i8_i64 failed ({rc})")
        return C

    def gemm_bf16_f64(self, A: np.ndarray, B: np.ndarray, nthreads: int | None = None,
                      ldc_pad: int = 0) -> np.ndarray:
        """A, B: uint16 arrays holding bf16 bit patterns.  Returns fp64 C."""
        assert A.dtype == np.uint16 and B.dtype == np.uint16 and A.shape[1] == B.shape[0]
        M, K = A.shape
        N = B.shape[1]
        C, buf, ldc = self._out(M, N, np.float64, ldc_pad)
        rc = self.lib.oracle_gemm_bf16_f64(M, N, K, A.ctypes.data, self._ld(A) if M and K else max(K, 1),
                                           B.ctypes.data, self._ld(B) if K and N else max(N, 1),
                                           buf.ctypes.data, ldc, self.threads(nthreads))
        if rc != 0:
            raise RuntimeError(f"oracle_gemm_bf16_f64 failed ({rc})")
        return C

    # -- column-major B ------------------------------------------------------
    @staticmethod
    def _from_bt(Bt: np.ndarray) -> np.ndarray:
        """B (K x N, row-major) from Bt (N x K): B[k][j] = Bt[j][k]."""
        assert Bt.ndim == 2
        B = np.empty((Bt.shape[1], Bt.shape[0]), dtype=Bt.dtype)   # fresh row-major buffer
        B[...] = Bt.T
        return B

    def gemm_i8_i32_bt(self, A: np.ndarray, Bt: np.ndarray, nthreads: int | None = None):
        """C = A @ Bt^T (int8, Bt is N x K).  Returns (C int32 M x N, overflow_count)."""
        return self.gemm_i8_i32(A, self._from_bt(Bt), nthreads)

    def gemm_bf16_f64_bt(self, A: np.ndarray, Bt: np.ndarray, nthreads: int | None = None) -> np.ndarray:
        """C = A @ Bt^T (bf16 bits, Bt is N x K).  Returns fp64 C."""
        return self.gemm_bf16_f64(A, self._from_bt(Bt), nthreads)

    def freivalds_i8_i32_bt(self, A: np.ndarray, Bt: np.ndarray, C: np.ndarray,
                            trials: int = 2, seed: int = 1234) -> int:
        return self.freivalds_i8_i32(A, self._from_bt(Bt), C, trials, seed)

    def bf16_to_double(self, bits: int) -> float:
        return float(self.lib.oracle_bf16_to_double(int(bits)))

    def freivalds_i8_i32(self, A: np.ndarray, B: np.ndarray, C: np.ndarray,
                         trials: int = 2, seed: int = 1234) -> int:
        """Number of (trial, row) pairs where A(Br) != Cr (0 = consistent)."""
        assert C.dtype == np.int32
        M, K = A.shape
        N = B.shape[1]
        bad = self.lib.oracle_freivalds_i8_i32(M, N, K, A.ctypes.data, self._ld(A) if M and K else max(K, 1),
                                               B.ctypes.data, self._ld(B) if K and N else max(N, 1),
                                               C.ctypes.data, self._ld(C) if M and N else max(N, 1),
                                               trials, seed)
        if bad < 0:
            raise RuntimeError(f"oracle_freivalds_i8_i32 failed ({bad})")
        return int(bad)


    # -- reduced-precision outputs ---------------------------------------------
    def requant_i32(self, C: np.ndarray, shift: int, bits: int) -> np.ndarray:
        """int32 results -> int8 (bits 8) or int16 (bits 16): C / 2^shift rounded to
        nearest, ties to even, then saturated."""
        src = np.ascontiguousarray(C, dtype=np.int32)
        out = np.empty(src.shape, dtype=np.int32)
        rc = self.lib.oracle_requant_i32(src.ctypes.data, src.size, int(shift), int(bits), out.ctypes.data)
        if rc != 0:
            raise RuntimeError(f"oracle_requant_i32 failed ({rc})")
        return out.astype(np.int8 if bits == 8 else np.int16)

    def round_bf16(self, C: np.ndarray) -> np.ndarray:
        """fp64 values -> nearest bf16 (ties to even), as uint16 bit patterns."""
        src = np.ascontiguousarray(C, dtype=np.float64)
        out = np.empty(src.shape, dtype=np.uint16)
        rc = self.lib.oracle_round_bf16(src.ctypes.data, src.size, out.ctypes.data)
        if rc != 0:
            raise RuntimeError(f"oracle_round_bf16 failed ({rc})")
        return out

    def bf16_from_double(self, x: float) -> int:
        return int(self.lib.oracle_bf16_from_double(float(x)))


_default: Oracle | None = None


def get() -> Oracle:
    """The default oracle build (compiled on first use if absent)."""
    global _default
    if _default is None:
        if not os.path.exists(LIB):
            build()
        _default = Oracle(LIB)
    return _default


def normalized_error(C: np.ndarray, C_ref: np.ndarray, K: int, amax_a: float, amax_b: float) -> float:
    """max|C - C_ref| / (K * max|A| * max|B|), the bf16 parity metric.

    With a zero denominator (K == 0 or an all-zero operand) the exact result is
    0 and the metric is 0 if C == 0 everywhere, else inf.
    """
    diff = float(np.max(np.abs(C.astype(np.float64) - C_ref))) if C.size else 0.0
    denom = float(K) * float(amax_a) * float(amax_b)
    if denom == 0.0:
        return 0.0 if diff == 0.0 else float("inf")
    return diff / denom
