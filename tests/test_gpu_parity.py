"""GPU path vs the CPU oracle, through the C ABI (needs an MI355X).

int8 -> int32 is compared element for element (bit-exact).  bf16 -> fp32 must
satisfy max|C - C_ref| / (K * max|A| * max|B|) <= 1e-5, and on integer-valued
bf16 operands (where every fp32 partial sum is exact in any order) it must be
exact.  Full-size workloads: int8 element for element against the whole oracle
product (plus Freivalds' test); bf16 on the whole C where the fp64 oracle takes
seconds, else on sampled rows, and exactly (Freivalds over the whole C) on
integer-valued operands.
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
NUM_CONFIGS = 41
GENERIC_CONFIGS = (0, 1)
GEMV_CONFIGS = (26, 27)      # M = 1 only: tests/test_gpu_gemv.py
TILE_CONFIGS = [c for c in range(NUM_CONFIGS) if c not in GEMV_CONFIGS]
RING_CONFIGS = [c for c in range(16, NUM_CONFIGS) if c not in GEMV_CONFIGS]


@pytest.fixture(autouse=True)
def _reset_plan():
    g.unforce()
    yield
    g.unforce()


def _inputs(dtype, M, N, K, seed):
    return inputs.make_inputs("int8" if dtype == I8 else "bf16", M, N, K, seed=seed)


def _check(dtype, A, B, C):
    (g.check_i8 if dtype == I8 else g.check_bf16)(A, B, C)


def test_native_library_is_the_path():
    assert torch.cuda.is_available()
    lib = b.lib()
    maps = open("/proc/self/maps").read()
    assert b.LIB_PATH in maps, "libgemm_mi355x.so is not mapped into this process"
    assert "gfx950" in b.gemm_version()
    assert lib is not None


# Shapes every vectorised config accepts (row strides K and N a multiple of 16
# bytes for both dtypes), ragged in M, N and K against every tile size.
VEC_SHAPES = [(1, 16, 16), (37, 48, 48), (64, 256, 128), (300, 272, 1040), (257, 528, 2064),
              (513, 784, 784)]
# Shapes only the element-wise (generic) loaders accept.
ODD_SHAPES = [(1, 1, 1), (3, 5, 7), (17, 13, 31), (65, 63, 129), (129, 255, 257), (70, 300, 1001)]


@pytest.mark.parametrize("split,reduce", [(1, -1), (3, 0), (3, 1), (3, 2)], ids=["s1", "s3sep", "s3fused", "s3atomic"])
@pytest.mark.parametrize("config", TILE_CONFIGS)
@pytest.mark.parametrize("dtype", [I8, BF], ids=["i8", "bf16"])
def test_every_config_matches_oracle(dtype, config, split, reduce):
    g.force(dtype, b.GEMM_KERNEL_AUTO, config, split, reduce)
    for i, (M, N, K) in enumerate(VEC_SHAPES):
        A, B = _inputs(dtype, M, N, K, seed=100 + i)
        print(f"dtype={dtype} config={config} split={split} reduce={reduce} shape={(M, N, K)}", flush=True)
        _check(dtype, A, B, g.gemm_gpu(dtype, A, B))
    for i, (M, N, K) in enumerate(ODD_SHAPES):
        A, B = _inputs(dtype, M, N, K, seed=200 + i)
        if config in GENERIC_CONFIGS:
            print(f"dtype={dtype} config={config} split={split} odd shape={(M, N, K)}", flush=True)
            _check(dtype, A, B, g.gemm_gpu(dtype, A, B))
        else:
            dA, lda = g.to_dev(A)
            dB, ldb = g.to_dev(B)
            dC, ldc = g.out_buffer(M, N, dtype)
            assert g.call(dtype, M, N, K, dA, lda, dB, ldb, dC, ldc) == b.GEMM_ERR_UNSUPPORTED


@pytest.mark.parametrize("config", [c for c in range(41) if c not in (26, 27)])
def test_bf16_integer_valued_is_exact(config):
    """Integer-valued bf16 in [-8, 8]: the fp32 result is exact whatever the order."""
    M, N, K = 200, 264, 4096
    A = inputs.small_int_bf16_matrix(M, K, seed=7)
    B = inputs.small_int_bf16_matrix(K, N, seed=8)
    for split in (1, 5):
        g.force(BF, b.GEMM_KERNEL_AUTO, config, split)
        C = g.gemm_gpu(BF, A, B)
        ref = oracle.get().gemm_bf16_f64(A, B)
        assert np.array_equal(C.astype(np.float64), ref), (config, split)


@pytest.mark.parametrize("dtype,M,K,N", inputs.SMALL, ids=[f"{c[0]}-{c[1]}" for c in inputs.SMALL])
def test_small_workloads_full_oracle(dtype, M, K, N):
    d = I8 if dtype == "int8" else BF
    A, B = inputs.make_inputs(dtype, M, N, K, seed=0)
    _check(d, A, B, g.gemm_gpu(d, A, B))


def _sampled_rows(M, seed=5):
    rng = np.random.default_rng(seed)
    rows = {0, M - 1, M // 2}
    rows.update(int(x) for x in rng.integers(0, M, size=5))
    return sorted(r for r in rows if 0 <= r < M)


BIG = inputs.SQUARE + inputs.RECT + inputs.SKINNY


# bf16 workloads up to this many multiply-adds are compared with the whole fp64 oracle
# product (seconds on the host); larger ones on sampled rows.
BF16_FULL_MACS = 10 ** 11


@pytest.mark.parametrize("dtype,M,K,N", BIG, ids=[f"{c[0]}-{c[1]}x{c[2]}x{c[3]}" for c in BIG])
def test_full_size_workloads(dtype, M, K, N):
    """Full-size workload with the selector's plan (the configuration the benchmark times),
    the same seeded inputs as the benchmark.  int8: the whole C element by element against
    the whole oracle product (and Freivalds' test over it).  bf16: the whole C against the
    fp64 oracle by the normalised error where that takes seconds, else sampled rows."""
    d = I8 if dtype == "int8" else BF
    fake = 1 << 40   # plan only: addresses are never dereferenced
    plan = b.gemm_plan(d, M, N, K, K, N, N, fake, 2 * fake, 3 * fake)
    print(f"full-size {dtype} M={M} K={K} N={N} plan={plan['name']} split={plan['split_k']}", flush=True)
    A, B = inputs.make_inputs(dtype, M, N, K, seed=0)
    C = g.gemm_gpu(d, A, B)
    o = oracle.get()
    full = d == I8 or M * N * K <= BF16_FULL_MACS
    rows = list(range(M)) if full else _sampled_rows(M)
    Ar = A if full else np.ascontiguousarray(A[rows])
    if d == I8:
        assert o.freivalds_i8_i32(A, B, np.ascontiguousarray(C), trials=2) == 0
        ref, ovf = o.gemm_i8_i32(Ar, B)
        assert ovf == 0
        bad = np.argwhere(C[rows] != ref)
        assert bad.size == 0, f"{len(bad)} mismatches, first {bad[:3].tolist()}"
    else:
        ref = o.gemm_bf16_f64(Ar, B)
        amax_a = float(np.max(np.abs(inputs.f32_from_bf16_bits(A))))
        amax_b = float(np.max(np.abs(inputs.f32_from_bf16_bits(B))))
        err = oracle.normalized_error(C[rows], ref, K, amax_a, amax_b)
        assert err <= g.BF16_TOL, err
        assert np.all(np.isfinite(C))


@pytest.mark.parametrize("M,K,N", [(s[1], s[2], s[3]) for s in BIG if s[0] == "bf16"],
                         ids=[f"{s[1]}x{s[2]}x{s[3]}" for s in BIG if s[0] == "bf16"])
def test_full_size_bf16_integer_valued_freivalds(M, K, N):
    """bf16 kernels at full size on integer-valued operands: the exact product, checked on
    the whole C by Freivalds in exact integer arithmetic (values in [-8, 8] fit int8)."""
    A = inputs.small_int_bf16_matrix(M, K, seed=11)
    B = inputs.small_int_bf16_matrix(K, N, seed=12)
    C = g.gemm_gpu(BF, A, B)
    Ci = C.astype(np.int64)
    assert np.array_equal(Ci.astype(np.float32), C), "non-integer output"
    A8 = inputs.f32_from_bf16_bits(A).astype(np.int8)
    B8 = inputs.f32_from_bf16_bits(B).astype(np.int8)
    assert oracle.get().freivalds_i8_i32(A8, B8, np.ascontiguousarray(Ci.astype(np.int32)), trials=2) == 0


@pytest.mark.parametrize("dtype", [I8, BF], ids=["i8", "bf16"])
def test_k_zero_writes_zeros_and_keeps_padding(dtype):
    M, N = 33, 40
    dA, _ = g.to_dev(np.zeros((M, 1), np.int8 if dtype == I8 else np.uint16))
    dB, _ = g.to_dev(np.zeros((1, N), np.int8 if dtype == I8 else np.uint16))
    sentinel = 777 if dtype == I8 else 7.5
    dC, ldc = g.out_buffer(M, N, dtype, pad_cols=5, sentinel=sentinel)
    assert g.call(dtype, M, N, 0, dA, 1, dB, N, dC, ldc) == b.GEMM_OK
    torch.cuda.synchronize()
    host = dC.cpu().numpy()
    C = host[: M * ldc].reshape(M, ldc)
    assert (C[:, :N] == 0).all()
    assert (C[:, N:] == sentinel).all() and (host[M * ldc:] == sentinel).all()


@pytest.mark.parametrize("dtype", [I8, BF], ids=["i8", "bf16"])
@pytest.mark.parametrize("pad,offs", [((16, 16, 16), (0, 0, 0)),      # aligned padding: vector path
                                      ((3, 5, 7), (0, 0, 0)),         # odd strides: generic path
                                      ((0, 0, 0), (1, 3, 0)),         # misaligned starts: generic
                                      ((32, 8, 1), (16, 16, 0))])
def test_strides_offsets_and_canaries(dtype, pad, offs):
    M, N, K = 150, 136, 272
    A, B = _inputs(dtype, M, N, K, seed=3)
    dA, lda = g.to_dev(A, pad[0], offs[0])
    dB, ldb = g.to_dev(B, pad[1], offs[1])
    sentinel = -99 if dtype == I8 else -0.25
    dC, ldc = g.out_buffer(M, N, dtype, pad[2], sentinel=sentinel)
    assert g.call(dtype, M, N, K, dA, lda, dB, ldb, dC, ldc, offs[0], offs[1], 0) == b.GEMM_OK
    torch.cuda.synchronize()
    host = dC.cpu().numpy()
    C = host[: M * ldc].reshape(M, ldc)
    _check(dtype, A, B, np.ascontiguousarray(C[:, :N]))
    assert (C[:, N:] == sentinel).all(), "row padding of C was written"
    assert (host[M * ldc:] == sentinel).all(), "memory past C was written"


def test_int8_split_k_is_invariant():
    M, N, K = 96, 512, 4096
    A, B = _inputs(I8, M, N, K, seed=9)
    outs = []
    for split in (1, 2, 5, 16, 32):
        for config, reduce in ((3, -1), (3, b.GEMM_REDUCE_ATOMIC), (28, b.GEMM_REDUCE_ATOMIC_FLAG)):
            g.force(I8, b.GEMM_KERNEL_AUTO, config, split, reduce)
            outs.append(g.gemm_gpu(I8, A, B))
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])
    g.check_i8(A, B, outs[0])


@pytest.mark.parametrize("config", [0, 3, 6, 8, 10, 12, 14, 15])
def test_split_k_reductions_agree_bitwise(config):
    """The in-kernel (last slice of each tile) and the separate reduction sum the K slices in
    the same fixed order: bf16 results are bit-identical between them and across calls,
    including split factors above the sixteen slices one reduction pass loads."""
    M, N, K = 70, 600, 8192
    A, B = _inputs(BF, M, N, K, seed=21)
    for split in (2, 7, 16, 17, 40):
        outs = []
        for reduce in (0, 1, 1, 0):
            g.force(BF, b.GEMM_KERNEL_AUTO, config, split, reduce)
            print(f"config={config} split={split} reduce={reduce}", flush=True)
            outs.append(g.gemm_gpu(BF, A, B).view(np.uint32))
        for o in outs[1:]:
            assert np.array_equal(o, outs[0]), (config, split)
        g.check_bf16(A, B, outs[0].view(np.float32))


def test_split_k_workspace_reuse_across_shapes_and_streams():
    """The per-stream workspace and its arrival counters are reused by every split-K call:
    growing and shrinking shapes, back-to-back calls without host synchronisation, and two
    streams in flight at once all give oracle-exact int8 results."""
    shapes = [(40, 512, 4096), (200, 1040, 2048), (8, 256, 8192), (300, 1536, 4096), (1, 48, 1024)]
    cases = []
    for i, (M, N, K) in enumerate(shapes):
        A, B = _inputs(I8, M, N, K, seed=40 + i)
        ref, _ = oracle.get().gemm_i8_i32(A, B)
        cases.append((M, N, K, A, B, ref))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    tile_plans = ((3, 6), (6, 16), (14, 5), (10, 3))
    ring_plans = ((28, 6), (31, 16), (20, 5), (38, 3))
    for reduce, plans in ((1, tile_plans), (0, tile_plans), (2, tile_plans), (3, ring_plans), (1, ring_plans)):
        for config, split in plans:
            g.force(I8, b.GEMM_KERNEL_AUTO, config, split, reduce)
            print(f"workspace reuse config={config} split={split} reduce={reduce}", flush=True)
            outs = []
            for rep in range(2):
                for j, (M, N, K, A, B, ref) in enumerate(cases):
                    st = streams[(j + rep) % 2]
                    dA, lda = g.to_dev(A)
                    dB, ldb = g.to_dev(B)
                    dC, ldc = g.out_buffer(M, N, I8)
                    torch.cuda.synchronize()
                    rc = b.gemm_i8_i32(M, N, K, dA.data_ptr(), lda, dB.data_ptr(), ldb, dC.data_ptr(), ldc,
                                       st.cuda_stream)
                    assert rc == b.GEMM_OK
                    outs.append((dA, dB, dC, ldc, M, N, ref))
            torch.cuda.synchronize()
            for dA, dB, dC, ldc, M, N, ref in outs:
                C = dC.cpu().numpy()[: M * ldc].reshape(M, ldc)[:, :N]
                assert np.array_equal(C, ref), (config, split, reduce, M, N)


@pytest.mark.parametrize("config,split,bt", [(28, 4, False), (31, 8, False), (30, 3, False), (14, 5, False),
                                             (10, 2, True), (20, 7, True), (0, 3, False)])
def test_int8_atomic_reduction(config, split, bt):
    """Atomic split-K reduction: C's M x N outputs are zeroed and every slice adds its
    partial tile into them.  Exact against the oracle on ragged shapes, the row padding
    and the memory around C untouched, and a second call into the same (now non-zero) C
    gives the same result."""
    g.force(I8, b.GEMM_KERNEL_AUTO, config, split, b.GEMM_REDUCE_ATOMIC)
    for M, N, K in [(75, 272, 2304), (1, 4112, 1024), (33, 48, 4096)]:
        A, B = _inputs(I8, M, N, K, seed=60 + M)
        Bx = np.ascontiguousarray(B.T) if bt else B
        p = b.gemm_plan(I8, M, N, K, K, K if bt else N, N + 5, 1 << 40, 2 << 40, 3 << 40, trans_b=bt)
        assert p["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC and p["workspace_bytes"] == 0, p
        dA, lda = g.to_dev(A)
        dB, ldb = g.to_dev(Bx)
        sentinel = -424242
        dC, ldc = g.out_buffer(M, N, I8, pad_cols=5, sentinel=sentinel)
        ref, ovf = oracle.get().gemm_i8_i32(A, B)
        assert ovf == 0
        for rep in range(2):
            print(f"atomic reduce config={config} split={split} bt={bt} shape={(M, N, K)} rep={rep}", flush=True)
            fn = g.call_bt if bt else g.call
            assert fn(I8, M, N, K, dA, lda, dB, ldb, dC, ldc) == b.GEMM_OK
            torch.cuda.synchronize()
            host = dC.cpu().numpy()
            C = host[: M * ldc].reshape(M, ldc)
            assert np.array_equal(C[:, :N], ref), np.argwhere(C[:, :N] != ref)[:3].tolist()
            assert (C[:, N:] == sentinel).all(), "row padding of C was written"
            assert (host[M * ldc:] == sentinel).all(), "memory past C was written"


@pytest.mark.parametrize("config", RING_CONFIGS)
def test_int8_atomic_flag_every_ring_config(config):
    """Atomic split-K reduction with C zeroed inside the GEMM by each tile's first K slice,
    whose signal the other slices wait for before adding.  Exact against the oracle on
    ragged shapes and split factors, with slices longer and shorter than the lead at which
    the signal is read, C's row pitch N + 5 and N; the row padding and the memory past C
    untouched; a second call into the same (now non-zero) C gives the same result."""
    for split in (2, 3, 9):
        g.force(I8, b.GEMM_KERNEL_AUTO, config, split, b.GEMM_REDUCE_ATOMIC_FLAG)
        for M, N, K in [(75, 272, 2304), (1, 4112, 1024), (33, 48, 4096), (300, 528, 640)]:
            A, B = _inputs(I8, M, N, K, seed=70 + M + split)
            p = b.gemm_plan(I8, M, N, K, K, N, N + 5, 1 << 40, 2 << 40, 3 << 40)
            assert p["split_k"] > 1 and p["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC_FLAG, p
            assert p["workspace_bytes"] == 0, p
            dA, lda = g.to_dev(A)
            dB, ldb = g.to_dev(B)
            sentinel = -515151
            ref, ovf = oracle.get().gemm_i8_i32(A, B)
            assert ovf == 0
            for pad, rep in ((5, 0), (5, 1), (0, 0), (0, 1)):
                if rep == 0:
                    dC, ldc = g.out_buffer(M, N, I8, pad_cols=pad, sentinel=sentinel)
                print(f"atomic flag config={config} split={split} shape={(M, N, K)} ldc={ldc} rep={rep}", flush=True)
                assert g.call(I8, M, N, K, dA, lda, dB, ldb, dC, ldc) == b.GEMM_OK
                torch.cuda.synchronize()
                host = dC.cpu().numpy()
                C = host[: M * ldc].reshape(M, ldc)
                assert np.array_equal(C[:, :N], ref), np.argwhere(C[:, :N] != ref)[:3].tolist()
                assert (C[:, N:] == sentinel).all(), "row padding of C was written"
                assert (host[M * ldc:] == sentinel).all(), "memory past C was written"


def test_release_workspace_then_reuse():
    M, N, K = 48, 512, 4096
    A, B = _inputs(I8, M, N, K, seed=50)
    for reduce in (1, 0):
        g.force(I8, b.GEMM_KERNEL_AUTO, 14, 8, reduce)
        g.check_i8(A, B, g.gemm_gpu(I8, A, B))
        assert b.gemm_release_workspace() == b.GEMM_OK
        assert b.gemm_release_workspace() == b.GEMM_OK      # nothing left: still fine
        g.check_i8(A, B, g.gemm_gpu(I8, A, B))


def test_bf16_split_k_is_reproducible():
    M, N, K = 96, 512, 4096
    A, B = _inputs(BF, M, N, K, seed=10)
    g.force(BF, b.GEMM_KERNEL_AUTO, 6, 7)
    c1 = g.gemm_gpu(BF, A, B)
    c2 = g.gemm_gpu(BF, A, B)
    assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32))
    g.check_bf16(A, B, c1)


@pytest.mark.parametrize("config", [2, 3, 6, 0, 8, 9, 10, 11, 12, 13, 14, 15, 16, 17, 18, 19, 20, 21, 22, 23, 24, 25, 28, 29, 30, 31, 32, 33, 34, 35, 36, 37, 38, 39, 40])
def test_int8_extremes_largest_k(config):
    """(-128)(-128) over K = 14336 is 234,881,024, the largest sum of the workload sweep."""
    g.force(I8, b.GEMM_KERNEL_AUTO, config, 0)
    M, N, K = 64, 256, 14336
    A = np.full((M, K), -128, np.int8)
    B = np.full((K, N), -128, np.int8)
    C = g.gemm_gpu(I8, A, B)
    assert (C == 234881024).all()
    B[:, ::2] = 127
    C = g.gemm_gpu(I8, A, B)
    assert (C[:, ::2] == -16256 * K).all() and (C[:, 1::2] == 234881024).all()


SPLIT_REDUCTIONS = [(3, 1, -1), (3, 4, b.GEMM_REDUCE_SEPARATE), (3, 4, b.GEMM_REDUCE_LAST_SLICE),
                    (3, 4, b.GEMM_REDUCE_ATOMIC), (3, 2, b.GEMM_REDUCE_ATOMIC), (28, 4, b.GEMM_REDUCE_ATOMIC_FLAG),
                    (28, 2, b.GEMM_REDUCE_ATOMIC_FLAG)]   # (config, split, reduction)


def test_int8_wraps_past_int32():
    """K = 131072 of (-128)(-128) = 2^31: documented to wrap modulo 2^32, like the oracle, with
    every split-K reduction."""
    M, N, K = 32, 64, 131072
    A = np.full((M, K), -128, np.int8)
    B = np.full((K, N), -128, np.int8)
    ref, ovf = oracle.get().gemm_i8_i32(A[:1], B[:, :1])
    assert ovf == 1
    for config, split, reduce in SPLIT_REDUCTIONS:
        g.force(I8, b.GEMM_KERNEL_AUTO, config, split, reduce)
        C = g.gemm_gpu(I8, A, B)
        assert (C == ref[0, 0]).all(), (config, split, reduce, np.unique(C)[:4])


def test_int8_partials_wrap_total_fits():
    """K = 262144: the first half of the products are (-128)(-128), the second (127)(-128).
    The running sum passes 2^31 halfway (a one-slice accumulator and the first slice's
    partial wrap) and the total, 131072 * 128 = 2^24, fits: modulo-2^32 arithmetic must still
    give it exactly, with every split and reduction."""
    M, N, K = 32, 64, 262144
    A = np.full((M, K), -128, np.int8)
    A[:, K // 2:] = 127
    B = np.full((K, N), -128, np.int8)
    ref, ovf = oracle.get().gemm_i8_i32(A[:1], B[:, :1])
    assert ovf == 0 and int(ref[0, 0]) == 2 ** 24
    for config, split, reduce in SPLIT_REDUCTIONS:
        g.force(I8, b.GEMM_KERNEL_AUTO, config, split, reduce)
        C = g.gemm_gpu(I8, A, B)
        assert (C == 2 ** 24).all(), (config, split, reduce, np.unique(C)[:4])


def test_torch_helpers():
    M, N, K = 130, 264, 520
    A, B = inputs.make_inputs("int8", M, N, K, seed=1)
    tA, tB = torch.from_numpy(A).to(g.DEV), torch.from_numpy(B).to(g.DEV)
    C = b.mm_i8_i32(tA, tB)
    g.check_i8(A, B, C.cpu().numpy())
    A, B = inputs.make_inputs("bf16", M, N, K, seed=2)
    tA = torch.from_numpy(A.view(np.int16)).to(g.DEV).view(torch.bfloat16)
    tB = torch.from_numpy(B.view(np.int16)).to(g.DEV).view(torch.bfloat16)
    C = b.mm_bf16_f32(tA, tB)
    g.check_bf16(A, B, C.cpu().numpy())
    with pytest.raises(TypeError):
        b.mm_i8_i32(tA, tB)
