"""Error paths of the C ABI that need a GPU: a split-K workspace that cannot be allocated
returns GEMM_ERR_NO_MEMORY with nothing queued and C untouched, and the next call, with
allocation possible again, runs normally (also for the atomic reduction whose C is zeroed
by the first slice: it needs per-tile counters); the atomic reduction with a fill kernel,
which needs no workspace, is unaffected (needs an MI355X)."""
import numpy as np
import pytest
import torch

from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import inputs
import gpu_helpers as g

pytestmark = pytest.mark.gpu
I8, BF = g.I8, g.BF
HOOK = "GEMM_MI355X_TEST_FAIL_WORKSPACE"


@pytest.fixture(autouse=True)
def _reset():
    g.unforce()
    yield
    g.unforce()


def _call(fn, A, B, sentinel):
    M, K = A.shape
    N = B.shape[1]
    dA, lda = g.to_dev(A)
    dB, ldb = g.to_dev(B)
    d = I8 if A.dtype == np.int8 else BF
    dC, ldc = g.out_buffer(M, N, d, 0, sentinel=sentinel)
    st = torch.cuda.current_stream().cuda_stream
    rc = fn(M, N, K, dA.data_ptr(), lda, dB.data_ptr(), ldb, dC.data_ptr(), ldc, st)
    torch.cuda.synchronize()
    return rc, dC.cpu().numpy()[: M * ldc].reshape(M, ldc)[:, :N]


@pytest.mark.parametrize("config,split,reduce", [(30, 8, 0), (28, 4, 1), (28, 4, 3)],
                         ids=["separate-reduce", "in-kernel", "atomic-flag-counters"])
def test_workspace_failure_then_recovery(monkeypatch, config, split, reduce):
    M, K, N = 64, 4096, 2048
    A, B = inputs.make_inputs("int8", M, N, K, seed=9)
    g.force(I8, b.GEMM_KERNEL_AUTO, config, split, reduce)
    assert b.gemm_release_workspace() == b.GEMM_OK      # the next split-K call must allocate
    monkeypatch.setenv(HOOK, "1")
    rc, C = _call(b.gemm_i8_i32, A, B, -5)
    assert rc == b.GEMM_ERR_NO_MEMORY, b.gemm_status_string(rc)
    assert (C == -5).all(), "a refused call wrote C"
    # plans without split-K, and the entry point that allocates nothing, are unaffected
    g.unforce()
    Ab, Bb = inputs.make_inputs("bf16", 16, 4096, 14336, seed=10)
    rc, Cb = _call(b.gemm_bf16_f32_noalloc, Ab, Bb, -5.0)
    assert rc == b.GEMM_OK
    assert g.bf16_error(Ab, Bb, Cb) <= g.BF16_TOL
    monkeypatch.delenv(HOOK)
    g.force(I8, b.GEMM_KERNEL_AUTO, config, split, reduce)
    rc, C = _call(b.gemm_i8_i32, A, B, -5)
    assert rc == b.GEMM_OK, b.gemm_status_string(rc)
    g.check_i8(A, B, C)


def test_atomic_reduction_needs_no_workspace(monkeypatch):
    """The atomic split-K reduction adds into C and allocates nothing: with every workspace
    allocation failing it still runs, exactly."""
    M, K, N = 64, 4096, 2048
    A, B = inputs.make_inputs("int8", M, N, K, seed=11)
    g.force(I8, b.GEMM_KERNEL_AUTO, 30, 8, b.GEMM_REDUCE_ATOMIC)
    assert b.gemm_release_workspace() == b.GEMM_OK
    monkeypatch.setenv(HOOK, "1")
    rc, C = _call(b.gemm_i8_i32, A, B, -5)
    assert rc == b.GEMM_OK, b.gemm_status_string(rc)
    g.check_i8(A, B, C)
