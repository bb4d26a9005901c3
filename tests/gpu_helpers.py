"""Helpers shared by the GPU tests: device buffers, calls through the C ABI, and
comparisons with the CPU oracle (int8 bit-exact; bf16 normalized error)."""
from __future__ import annotations

import numpy as np
import torch

from oracle import oracle
from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import inputs

DEV = torch.device("cuda:0")
BF16_TOL = 1e-5     # max|C - C_ref| / (K * max|A| * max|B|)
I8, BF = b.GEMM_DTYPE_I8_I32, b.GEMM_DTYPE_BF16_F32


def to_dev(x: np.ndarray, pad_cols: int = 0, offset_elems: int = 0) -> tuple[torch.Tensor, int]:
    """Copies a 2-D int8 / uint16(bf16 bits) array to the GPU.  Returns (buffer, ld):
    the matrix starts `offset_elems` into the buffer with row stride cols + pad_cols."""
    rows, cols = x.shape
    ld = cols + pad_cols
    host = x.view(np.int16) if x.dtype == np.uint16 else x
    flat = np.zeros(offset_elems + rows * ld + 64, dtype=host.dtype)
    if rows and cols:
        flat[offset_elems: offset_elems + rows * ld].reshape(rows, ld)[:, :cols] = host
    return torch.from_numpy(flat).to(DEV), ld


def out_buffer(M: int, N: int, dtype: int, pad_cols: int = 0, sentinel=None):
    ld = N + pad_cols
    tdt = torch.int32 if dtype == I8 else torch.float32
    buf = torch.empty(M * ld + 128, dtype=tdt, device=DEV)
    if sentinel is None:
        sentinel = -123456789 if dtype == I8 else float("nan")
    buf.fill_(sentinel)
    return buf, ld


def call(dtype: int, M: int, N: int, K: int, A, lda, B, ldb, C, ldc, a_off=0, b_off=0, c_off=0) -> int:
    fn = b.gemm_i8_i32 if dtype == I8 else b.gemm_bf16_f32
    e = 1 if dtype == I8 else 2
    stream = torch.cuda.current_stream().cuda_stream
    return fn(M, N, K, A.data_ptr() + a_off * e, lda, B.data_ptr() + b_off * e, ldb,
              C.data_ptr() + c_off * 4, ldc, stream)


def gemm_gpu(dtype: int, A: np.ndarray, B: np.ndarray, pad=(0, 0, 0), offs=(0, 0, 0)) -> np.ndarray:
    """Runs the library on host arrays and returns C (M x N) as numpy."""
    M, K = A.shape
    N = B.shape[1]
    dA, lda = to_dev(A, pad[0], offs[0])
    dB, ldb = to_dev(B, pad[1], offs[1])
    dC, ldc = out_buffer(M, N, dtype, pad[2])
    rc = call(dtype, M, N, K, dA, max(lda, 1), dB, max(ldb, 1), dC, max(ldc, 1), offs[0], offs[1], 0)
    assert rc == b.GEMM_OK, b.gemm_status_string(rc)
    torch.cuda.synchronize()
    host = dC.cpu().numpy()
    if M == 0 or N == 0:
        return np.zeros((M, N), host.dtype)
    return host[: M * ldc].reshape(M, ldc)[:, :N]


def check_i8(A: np.ndarray, B: np.ndarray, C: np.ndarray) -> None:
    ref, ovf = oracle.get().gemm_i8_i32(A, B)
    assert ovf == 0
    bad = np.argwhere(C != ref)
    assert bad.size == 0, f"{len(bad)} mismatches, first {bad[:3].tolist()}: {C[tuple(bad[0])]} vs {ref[tuple(bad[0])]}"


def bf16_error(A: np.ndarray, B: np.ndarray, C: np.ndarray, ref: np.ndarray | None = None) -> float:
    if ref is None:
        ref = oracle.get().gemm_bf16_f64(A, B)
    amax_a = float(np.max(np.abs(inputs.f32_from_bf16_bits(A)))) if A.size else 0.0
    amax_b = float(np.max(np.abs(inputs.f32_from_bf16_bits(B)))) if B.size else 0.0
    assert np.all(np.isfinite(C)), "non-finite output"
    return oracle.normalized_error(C, ref, A.shape[1], amax_a, amax_b)


def check_bf16(A: np.ndarray, B: np.ndarray, C: np.ndarray) -> None:
    err = bf16_error(A, B, C)
    assert err <= BF16_TOL, err


def call_bt(dtype: int, M: int, N: int, K: int, A, lda, Bt, ldbt, C, ldc) -> int:
    fn = b.gemm_i8_i32_bt if dtype == I8 else b.gemm_bf16_f32_bt
    stream = torch.cuda.current_stream().cuda_stream
    return fn(M, N, K, A.data_ptr(), lda, Bt.data_ptr(), ldbt, C.data_ptr(), ldc, stream)


def gemm_gpu_bt(dtype: int, A: np.ndarray, Bt: np.ndarray, pad=(0, 0, 0)) -> np.ndarray:
    """Runs the column-major-B entry point (Bt is N x K) and returns C (M x N) as numpy."""
    M, K = A.shape
    N = Bt.shape[0]
    dA, lda = to_dev(A, pad[0])
    dB, ldbt = to_dev(Bt, pad[1])
    dC, ldc = out_buffer(M, N, dtype, pad[2])
    rc = call_bt(dtype, M, N, K, dA, max(lda, 1), dB, max(ldbt, 1), dC, max(ldc, 1))
    assert rc == b.GEMM_OK, b.gemm_status_string(rc)
    torch.cuda.synchronize()
    host = dC.cpu().numpy()
    if M == 0 or N == 0:
        return np.zeros((M, N), host.dtype)
    return host[: M * ldc].reshape(M, ldc)[:, :N]


def force(dtype: int, kernel: int = b.GEMM_KERNEL_AUTO, config: int = -1, split: int = 0,
          reduce: int = -1) -> None:
    assert b.gemm_force_plan(dtype, kernel, config, split) == b.GEMM_OK
    assert b.gemm_force_reduce(dtype, reduce) == b.GEMM_OK


def unforce() -> None:
    for d in (I8, BF):
        b.gemm_force_plan(d, b.GEMM_KERNEL_AUTO, -1, 0)
        b.gemm_force_reduce(d, -1)
