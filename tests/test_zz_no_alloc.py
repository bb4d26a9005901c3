"""gemm_bf16_f32_noalloc, the entry point that allocates nothing, against gemm_bf16_f32
through the C ABI (needs an MI355X): the same plan and kernels, so the same fp32 result
bit for bit, on split-K plans whose partials and counters live in the library's fixed
per-device scratch; two calls in a row, the second with a smaller input; a plan whose
partials exceed the scratch is refused before anything runs."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import inputs
import gpu_helpers as g

pytestmark = pytest.mark.gpu
BF = g.BF


@pytest.fixture(autouse=True)
def _reset_plan():
    g.unforce()
    yield
    g.unforce()


def _run(fn, A, B, pad=4):
    M, K = A.shape
    N = B.shape[1]
    dA, lda = g.to_dev(A)
    dB, ldb = g.to_dev(B)
    dC, ldc = g.out_buffer(M, N, BF, pad, sentinel=-7.0)
    st = torch.cuda.current_stream().cuda_stream
    rc = fn(M, N, K, dA.data_ptr(), lda, dB.data_ptr(), ldb, dC.data_ptr(), ldc, st)
    torch.cuda.synchronize()
    host = dC.cpu().numpy()
    full = host[: M * ldc].reshape(M, ldc)
    assert (full[:, N:] == -7.0).all() and (host[M * ldc:] == -7.0).all(), "wrote outside C"
    return rc, full[:, :N]


def _plan(M, N, K):
    # addresses only set the alignment class (never dereferenced); device buffers are 256-byte aligned
    return b.gemm_plan(BF, M, N, K, K, N, N, 0x10000000, 0x20000000, 0x40000000)


def test_noalloc_matches_gemm_bf16_f32_on_two_calls():
    # first a split-K plan reduced by a separate kernel, then a smaller one reduced in-kernel
    cases = [(16, 4096, 14336, 0), (1, 2048, 14336, 1)]
    for i, (M, N, K, reduce) in enumerate(cases):
        g.force(BF, b.GEMM_KERNEL_AUTO, 28, 4 + 2 * i, reduce)     # ring_32x256_w4_r4
        p = _plan(M, N, K)
        assert p["split_k"] == 4 + 2 * i and p["reduce_in_kernel"] == reduce, p
        A, B = inputs.make_inputs("bf16", M, N, K, seed=60 + i)
        print(f"noalloc call {i}: M={M} N={N} K={K} split={p['split_k']} reduce={reduce}", flush=True)
        rc0, C0 = _run(b.gemm_bf16_f32, A, B)
        rc1, C1 = _run(b.gemm_bf16_f32_noalloc, A, B)
        assert rc0 == b.GEMM_OK and rc1 == b.GEMM_OK, (rc0, rc1)
        assert np.array_equal(C0.view(np.uint32), C1.view(np.uint32)), "not bit-identical to gemm_bf16_f32"
        err = g.bf16_error(A, B, C1)
        assert err <= g.BF16_TOL, err


def test_noalloc_selector_plans_and_unsplit_shapes():
    # the selector's own plans (skinny split-K, and a square one with no scratch at all)
    for (M, K, N) in ((64, 14336, 4096), (1, 4096, 14336), (300, 272, 1040)):
        A, B = inputs.make_inputs("bf16", M, N, K, seed=M + N)
        print(f"noalloc selector plan: M={M} N={N} K={K} plan={_plan(M, N, K)['name']}", flush=True)
        rc0, C0 = _run(b.gemm_bf16_f32, A, B)
        rc1, C1 = _run(b.gemm_bf16_f32_noalloc, A, B)
        assert rc0 == b.GEMM_OK and rc1 == b.GEMM_OK, (rc0, rc1)
        assert np.array_equal(C0.view(np.uint32), C1.view(np.uint32))


def test_noalloc_refuses_a_plan_beyond_its_scratch():
    # 8 slices of 1024 x 1024 fp32 partials = 32 MiB > 16 MiB - 64 KiB: refused, C untouched;
    # the allocating entry point runs the same plan
    M = N = 1024
    K = 8192
    g.force(BF, b.GEMM_KERNEL_AUTO, 10, 8, 0)
    A, B = inputs.make_inputs("bf16", M, N, K, seed=3)
    rc, C = _run(b.gemm_bf16_f32_noalloc, A, B)
    assert rc == b.GEMM_ERR_SCRATCH_LIMIT, b.gemm_status_string(rc)
    assert (C == -7.0).all(), "refused call wrote C"
    rc, C = _run(b.gemm_bf16_f32, A, B)
    assert rc == b.GEMM_OK
    assert g.bf16_error(A, B, C) <= g.BF16_TOL
