"""Split-K GEMM calls captured in a HIP graph and replayed (needs an MI355X).

Every reduction leaves the stream's workspace as it found it (arrival counters and
credit counters back at zero, partial planes rewritten by each call), so a captured
call may be replayed any number of times.  Each case runs the call eagerly once on a
side stream (which also creates that stream's workspace, so the capture allocates
nothing), captures the same call into a graph, and replays the graph four times, with
other GEMMs on the same stream and workspace in between, each replay checked against
the eager result bit for bit (and that against the oracle).  The entry point that
allocates nothing is captured the same way.
"""
import numpy as np
import pytest
import torch

from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import inputs
import gpu_helpers as g

pytestmark = pytest.mark.gpu
I8, BF = g.I8, g.BF


@pytest.fixture(autouse=True)
def _reset_plan():
    g.unforce()
    yield
    g.unforce()


def _operands(dtype, M, N, K, seed):
    A, B = inputs.make_inputs("int8" if dtype == I8 else "bf16", M, N, K, seed=seed)
    dA, lda = g.to_dev(A)
    dB, ldb = g.to_dev(B)
    return A, B, dA, lda, dB, ldb


# (dtype, config, split, reduction): ring_32x256_w4_r4 = 28, ring_64x128_w4_r5 = 30,
# macro_128x256_w4 = 3 (whose atomic reduction zeroes C with a fill kernel)
CASES = [(I8, 28, 4, b.GEMM_REDUCE_ATOMIC_FLAG), (I8, 30, 8, b.GEMM_REDUCE_ATOMIC_FLAG),
         (I8, 3, 4, b.GEMM_REDUCE_ATOMIC), (I8, 28, 4, b.GEMM_REDUCE_LAST_SLICE),
         (I8, 30, 3, b.GEMM_REDUCE_SEPARATE), (BF, 28, 4, b.GEMM_REDUCE_LAST_SLICE),
         (BF, 30, 8, b.GEMM_REDUCE_SEPARATE)]


@pytest.mark.parametrize("dtype,config,split,reduce", CASES,
                         ids=["i8-flag4", "i8-flag8", "i8-fill", "i8-last", "i8-sep", "bf16-last", "bf16-sep"])
def test_graph_replays_match_eager(dtype, config, split, reduce):
    M, N, K = 48, 4112, 4096
    g.force(dtype, b.GEMM_KERNEL_AUTO, config, split, reduce)
    p = b.gemm_plan(dtype, M, N, K, K, N, N, 1 << 40, 2 << 40, 3 << 40)
    assert p["split_k"] == split and p["reduce_in_kernel"] == reduce, p
    A, B, dA, lda, dB, ldb = _operands(dtype, M, N, K, seed=80)
    A2, B2, dA2, _, dB2, _ = _operands(dtype, M, N, K, seed=81)       # the eager work between replays
    fn = b.gemm_i8_i32 if dtype == I8 else b.gemm_bf16_f32
    s = torch.cuda.Stream()
    dC, ldc = g.out_buffer(M, N, dtype)
    dC2, _ = g.out_buffer(M, N, dtype)

    def gemm(a, bb, c):
        return fn(M, N, K, a.data_ptr(), lda, bb.data_ptr(), ldb, c.data_ptr(), ldc, s.cuda_stream)

    torch.cuda.synchronize()
    print(f"graph eager dtype={dtype} config={config} split={split} reduce={reduce}", flush=True)
    assert gemm(dA, dB, dC) == b.GEMM_OK
    s.synchronize()
    eager = dC.cpu().numpy()[: M * ldc].reshape(M, ldc)[:, :N].copy()
    (g.check_i8 if dtype == I8 else g.check_bf16)(A, B, eager)

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        dC.fill_(-1)
    s.synchronize()
    print("graph capture", flush=True)
    with torch.cuda.graph(graph, stream=s):
        rc = gemm(dA, dB, dC)
    assert rc == b.GEMM_OK
    for rep in range(4):
        with torch.cuda.stream(s):
            dC.fill_(-2 - rep)
        print(f"graph replay {rep}", flush=True)
        graph.replay()
        torch.cuda.synchronize()
        got = dC.cpu().numpy()[: M * ldc].reshape(M, ldc)[:, :N]
        assert np.array_equal(got.view(np.uint32), eager.view(np.uint32)), f"replay {rep} differs"
        assert gemm(dA2, dB2, dC2) == b.GEMM_OK       # eager work on the same stream and workspace
        s.synchronize()
    other = dC2.cpu().numpy()[: M * ldc].reshape(M, ldc)[:, :N]
    (g.check_i8 if dtype == I8 else g.check_bf16)(A2, B2, other)


def test_graph_replays_noalloc():
    """gemm_bf16_f32_noalloc captured with a split-K plan (its counters cleared by a fill
    kernel inside the call, which the capture records) replays like the eager call."""
    M, N, K = 16, 4096, 14336
    g.force(BF, b.GEMM_KERNEL_AUTO, 20, 4, b.GEMM_REDUCE_LAST_SLICE)      # ring_32x64_w2
    A, B, dA, lda, dB, ldb = _operands(BF, M, N, K, seed=82)
    s = torch.cuda.Stream()
    dC, ldc = g.out_buffer(M, N, BF)

    def gemm():
        return b.gemm_bf16_f32_noalloc(M, N, K, dA.data_ptr(), lda, dB.data_ptr(), ldb, dC.data_ptr(), ldc,
                                       s.cuda_stream)

    torch.cuda.synchronize()
    assert gemm() == b.GEMM_OK
    s.synchronize()
    eager = dC.cpu().numpy()[: M * ldc].reshape(M, ldc)[:, :N].copy()
    g.check_bf16(A, B, eager)
    graph = torch.cuda.CUDAGraph()
    print("graph capture noalloc", flush=True)
    with torch.cuda.graph(graph, stream=s):
        rc = gemm()
    assert rc == b.GEMM_OK
    for rep in range(4):
        with torch.cuda.stream(s):
            dC.fill_(float(-3 - rep))
        print(f"graph replay noalloc {rep}", flush=True)
        graph.replay()
        torch.cuda.synchronize()
        got = dC.cpu().numpy()[: M * ldc].reshape(M, ldc)[:, :N]
        assert np.array_equal(got.view(np.uint32), eager.view(np.uint32)), f"replay {rep} differs"
