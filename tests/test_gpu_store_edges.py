"""The C epilogue's store forms at their edges, through the C ABI (needs an MI355X).

After the accumulators are transposed across groups of four lanes, a lane writes
four consecutive outputs of one row with a single store when C's pitch and start
allow it (ldc a multiple of 4, C aligned to four elements), else one by one; where
fewer than four columns remain (N % 4 != 0) the last ones also go out one by one.
The 4-wave 256 x 256 tiles (configuration 2 below) keep one output per store.
Exercised for every output type (int32, fp32, int8, int16, bf16) over pitches with
ldc % 4 = 0..3, C starting 0..3 elements past an aligned address, N % 4 = 0..3 and
ragged M, on one configuration of each kernel family, against the oracle: int8
bit-exact, bf16 on integer-valued operands (every fp32 partial sum is then exact,
so the fp32 result and its bf16 rounding are unique).  Sentinels fill the buffer
before C, the padding of each row and the space after C: nothing but the M x N
outputs may change.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import inputs
import gpu_helpers as g

pytestmark = pytest.mark.gpu
I8, BF = g.I8, g.BF

# kind: (element type of C, sentinel, entry point, entry point with column-major B)
KINDS = {
    "i32": (torch.int32, -123456789, "gemm_i8_i32", "gemm_i8_i32_bt"),
    "i8": (torch.int8, -77, "gemm_i8_i8", "gemm_i8_i8_bt"),
    "i16": (torch.int16, -7777, "gemm_i8_i16", "gemm_i8_i16_bt"),
    "f32": (torch.float32, -0.375, "gemm_bf16_f32", "gemm_bf16_f32_bt"),
    "bf16": (torch.int16, 0x7FC1, "gemm_bf16_bf16", "gemm_bf16_bf16_bt"),   # a quiet NaN
}
SHIFT = {"i8": 9, "i16": 3}
GUARD = 64      # sentinel elements before C


@pytest.fixture(autouse=True)
def _reset_plan():
    g.unforce()
    yield
    g.unforce()


def _operands(kind, M, N, K, seed, bt):
    if kind in ("i32", "i8", "i16"):
        A, B = inputs.make_inputs("int8", M, N, K, seed=seed)
    else:
        A = inputs.small_int_bf16_matrix(M, K, seed=seed)
        B = inputs.small_int_bf16_matrix(K, N, seed=seed + 1)
    return A, (np.ascontiguousarray(B.T) if bt else B)


def _expected(kind, A, Bx, bt):
    o = oracle.get()
    if kind in ("i32", "i8", "i16"):
        exact, ovf = o.gemm_i8_i32_bt(A, Bx) if bt else o.gemm_i8_i32(A, Bx)
        assert ovf == 0
        if kind == "i32":
            return exact.astype(np.int32)
        return o.requant_i32(exact, SHIFT[kind], 8 if kind == "i8" else 16)
    exact = o.gemm_bf16_f64_bt(A, Bx) if bt else o.gemm_bf16_f64(A, Bx)
    if kind == "f32":
        return exact.astype(np.float32)
    return o.round_bf16(exact).view(np.int16)


def _run(kind, A, Bx, N, pad, c_off, bt):
    """Calls the entry point of `kind` with C at `c_off` elements past GUARD sentinels and
    row pitch N + pad; returns (C, whole buffer, ldc)."""
    M, K = A.shape
    tdt, sentinel, name, name_bt = KINDS[kind]
    ldc = N + pad
    buf = torch.full((GUARD + c_off + M * ldc + GUARD,), sentinel, dtype=tdt, device=g.DEV)
    dA, lda = g.to_dev(A)
    dB, ldb = g.to_dev(Bx)
    esize = buf.element_size()
    c_ptr = buf.data_ptr() + (GUARD + c_off) * esize
    args = (M, N, K, dA.data_ptr(), lda, dB.data_ptr(), ldb, c_ptr, ldc)
    fn = getattr(b, name_bt if bt else name)
    st = torch.cuda.current_stream().cuda_stream
    rc = fn(*args, SHIFT[kind], st) if kind in SHIFT else fn(*args, st)
    assert rc == b.GEMM_OK, b.gemm_status_string(rc)
    torch.cuda.synchronize()
    host = buf.cpu().numpy()
    C = host[GUARD + c_off: GUARD + c_off + M * ldc].reshape(M, ldc)
    return C, host, ldc


def _check(kind, A, Bx, N, pad, c_off, bt):
    M = A.shape[0]
    C, host, ldc = _run(kind, A, Bx, N, pad, c_off, bt)
    ref = _expected(kind, A, Bx, bt)
    got = C[:, :N]
    if kind == "f32":
        bad = np.argwhere(~(got == ref))
    else:
        bad = np.argwhere(got != ref)
    assert bad.size == 0, f"{len(bad)} mismatches, first {bad[:3].tolist()}"
    sentinel = np.array(KINDS[kind][1], dtype=host.dtype)
    assert (C[:, N:] == sentinel).all(), "row padding of C was written"
    assert (host[: GUARD + c_off] == sentinel).all(), "memory before C was written"
    assert (host[GUARD + c_off + M * ldc:] == sentinel).all(), "memory after C was written"


# (ldc - N, C offset in elements): the wide form, then each way of losing it
LAYOUTS = [(0, 0), (4, 0), (1, 0), (2, 1), (3, 2), (0, 1), (0, 2), (0, 3), (4, 3)]


@pytest.mark.parametrize("kind", list(KINDS))
@pytest.mark.parametrize("config", [2, 6, 10, 14, 16, 20, 31])
def test_store_forms_row_major_b(kind, config):
    """Row-major B (N a multiple of 16, as the vector-load kernels need), every pitch and start."""
    M, N, K = 75, 144, 160
    dt = I8 if kind in ("i32", "i8", "i16") else BF
    g.force(dt, b.GEMM_KERNEL_AUTO, config, 1)
    A, B = _operands(kind, M, N, K, seed=1200 + config, bt=False)
    for pad, c_off in LAYOUTS:
        print(f"store edges: kind={kind} config={config} M={M} N={N} K={K} pad={pad} c_off={c_off}", flush=True)
        _check(kind, A, B, N, pad, c_off, bt=False)


@pytest.mark.parametrize("kind", list(KINDS))
@pytest.mark.parametrize("config", [0, 10, 16, 20, 31])
def test_store_forms_ragged_n(kind, config):
    """Column-major B lets the vector-load kernels take any N: N % 4 = 1, 2, 3, 0."""
    M, K = 75, 160
    dt = I8 if kind in ("i32", "i8", "i16") else BF
    g.force(dt, b.GEMM_KERNEL_AUTO, config, 1)
    for N in (141, 142, 143, 140, 33):
        A, Bt = _operands(kind, M, N, K, seed=1300 + N, bt=True)
        for pad, c_off in [(0, 0), (3, 0), (1, 1), (0, 2)]:
            print(f"store edges bt: kind={kind} config={config} M={M} N={N} K={K} pad={pad} c_off={c_off}", flush=True)
            _check(kind, A, Bt, N, pad, c_off, bt=True)
