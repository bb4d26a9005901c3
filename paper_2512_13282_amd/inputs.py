"""Seeded synthetic GEMM operands, shared by the tests, the benchmark and the smoke check.

This module holds no GEMM arithmetic: it only draws matrices.  Both the GPU
path and the CPU oracle consume what it returns.

Recipe (the paper benchmarks synthetic GEMM sizes and names no dataset):

* int8 : i.i.d. uniform integers in [-128, 127];
* bf16 : i.i.d. N(0, 1) float32 draws rounded to bf16, round-to-nearest-even,
  returned as raw uint16 bit patterns;
* A is drawn from ``numpy.random.default_rng(seed)`` and B from
  ``default_rng(seed + 1)`` (PCG64), both row-major and contiguous.
"""
from __future__ import annotations

import numpy as np

DTYPES = ("int8", "bf16")


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); uint16 bits out.  Infinities
    keep their sign; a NaN stays a NaN (its upper half with the quiet bit set)."""
    # In uint32: the sum stays below 2^32 for every non-NaN pattern (at most
    # 0xFF800000 + 0x8000); NaN sums may wrap, and are replaced.
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    one, half = np.uint32(1), np.uint32(0x7FFF)
    r = ((u + half + ((u >> np.uint32(16)) & one)) >> np.uint32(16)).astype(np.uint16)
    nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    if nan.any():
        r[nan] = ((u[nan] >> np.uint32(16)) | np.uint32(0x40)).astype(np.uint16)
    return r


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32 (for building test inputs)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def int8_matrix(rows: int, cols: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(-128, 128, size=(rows, cols), dtype=np.int8)


def bf16_matrix(rows: int, cols: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return bf16_bits_from_f32(rng.standard_normal(size=(rows, cols), dtype=np.float32))


def make_inputs(dtype: str, M: int, N: int, K: int, seed: int = 0):
    """Returns (A, B): A is M x K, B is K x N; int8 arrays or uint16 bf16 bits."""
    if dtype == "int8":
        return int8_matrix(M, K, seed), int8_matrix(K, N, seed + 1)
    if dtype == "bf16":
        return bf16_matrix(M, K, seed), bf16_matrix(K, N, seed + 1)
    raise ValueError(f"unknown dtype {dtype!r}")


def small_int_bf16_matrix(rows: int, cols: int, seed: int, lo: int = -8, hi: int = 8) -> np.ndarray:
    """bf16 matrix of integers in [lo, hi]: every fp32 partial sum of a GEMM over such
    operands is an integer below 2^24 while K * max|a| * max|b| < 2^24, so the exact
    result is reached in any summation order."""
    rng = np.random.default_rng(seed)
    v = rng.integers(lo, hi + 1, size=(rows, cols)).astype(np.float32)
    return bf16_bits_from_f32(v)


# Workloads of the paper-shaped sweep: (dtype, M, K, N).
SQUARE = [(d, s, s, s) for d in DTYPES for s in (2048, 4096, 8192)]
RECT = [(d, M, K, N) for d in DTYPES for (M, K, N) in ((2048, 4096, 11008), (2048, 11008, 4096),
                                                       (4096, 4096, 12288))]
SKINNY = [(d, M, K, N) for d in DTYPES for M in (1, 16, 64) for (K, N) in ((4096, 14336), (14336, 4096))]
SMALL = [("int8", 256, 256, 256), ("bf16", 1024, 1024, 1024)]
ALL_CONFIGS = SMALL + SQUARE + RECT + SKINNY
# For the plan tuner: decode batch sizes between the skinny workloads' 1, 16 and 64 rows,
# the skinny rows at the rectangle workloads' layer dimensions, and short prefill chunks
# (128 and 256 rows) at all five layer dimensions; then the same row counts at further
# transformer projection sizes (K = hidden size 4096 or 8192; N = the fused query/key/value
# width, the hidden size, or the feed-forward width, and the transposed feed-forward shape).
LAYER_KN = ((4096, 14336), (14336, 4096), (4096, 11008), (11008, 4096), (4096, 12288))
DECODE = ([(d, M, K, N) for d in DTYPES for M in (8, 32) for (K, N) in LAYER_KN[:2]] +
          [(d, M, K, N) for d in DTYPES for M in (1, 16, 32, 64) for (K, N) in LAYER_KN[2:]])
PREFILL = [(d, M, K, N) for d in DTYPES for M in (128, 256) for (K, N) in LAYER_KN]
MORE_LAYER_KN = ((4096, 6144), (4096, 4096), (8192, 28672), (28672, 8192), (8192, 10240), (8192, 8192))
MORE_LAYERS = [(d, M, K, N) for (K, N) in MORE_LAYER_KN for d in DTYPES for M in (1, 16, 64, 128, 256)]
# Longer prefill chunks (512 and 2048 rows) at all eleven sizes.
PREFILL_LONG = [(d, M, K, N) for (K, N) in LAYER_KN + MORE_LAYER_KN for d in DTYPES for M in (512, 2048)]
# Sizes that are not powers of two (hidden size 3584: feed-forward 18944 and its
# transpose, fused query/key/value 4608; hidden size 5120: 13824, its transpose and
# 15360), at every row count above.
ODD_LAYER_KN = ((3584, 18944), (18944, 3584), (3584, 4608), (5120, 13824), (13824, 5120), (5120, 15360))
ODD_LAYERS = [(d, M, K, N) for (K, N) in ODD_LAYER_KN for d in DTYPES for M in (1, 16, 64, 128, 256, 512, 2048)]
