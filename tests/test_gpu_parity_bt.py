"""GPU path vs the CPU oracle for B stored column-major (Bt, N x K), through the
*_bt entry points of the C ABI (needs an MI355X).  Same bars as the row-major
tests: int8 bit-exact, bf16 within 1e-5 normalised error and exact on
integer-valued operands; full sizes by Freivalds plus sampled oracle rows."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import inputs
import gpu_helpers as g

pytestmark = pytest.mark.gpu
I8, BF = g.I8, g.BF
BT_CONFIGS = (0, 1, 8, 9, 10, 11, 12, 16, 17, 18, 19, 20, 21, 22, 23, 24, 25, 28, 29, 30, 31, 32, 33, 34, 35, 36, 37, 38, 39, 40)
GENERIC_CONFIGS = (0, 1)


@pytest.fixture(autouse=True)
def _reset_plan():
    g.unforce()
    yield
    g.unforce()


def _inputs_bt(dtype, M, N, K, seed):
    """A (M x K) and Bt (N x K) from the same seeded generators as the row-major tests."""
    name = "int8" if dtype == I8 else "bf16"
    A, B = inputs.make_inputs(name, M, N, K, seed=seed)
    return A, np.ascontiguousarray(B.T)


def _check_bt(dtype, A, Bt, C):
    o = oracle.get()
    if dtype == I8:
        ref, ovf = o.gemm_i8_i32_bt(A, Bt)
        assert ovf == 0
        bad = np.argwhere(C != ref)
        assert bad.size == 0, f"{len(bad)} mismatches, first {bad[:3].tolist()}"
    else:
        ref = o.gemm_bf16_f64_bt(A, Bt)
        err = g.bf16_error(A, np.ascontiguousarray(Bt.T), C, ref)
        assert err <= g.BF16_TOL, err


# Shapes the vectorised column-major path accepts (K a multiple of 16 bytes; N free),
# ragged in M, N and K against every tile size.
VEC_SHAPES = [(1, 16, 16), (37, 45, 48), (64, 256, 128), (300, 270, 1040), (257, 529, 2064),
              (513, 784, 784)]
ODD_SHAPES = [(1, 1, 1), (3, 5, 7), (17, 13, 31), (65, 63, 129), (129, 255, 257), (70, 300, 1001)]


RING_BT_CONFIGS = [c for c in BT_CONFIGS if c >= 16]


@pytest.mark.parametrize("config", RING_BT_CONFIGS)
def test_int8_atomic_flag_bt(config):
    """Column-major B with the atomic split-K reduction whose C is zeroed by each tile's first
    K slice: exact against the oracle for every ring configuration, ragged N, two splits, C's
    row pitch unpadded and padded to a multiple of 4."""
    for split in (2, 5):
        g.force(I8, b.GEMM_KERNEL_AUTO, config, split, b.GEMM_REDUCE_ATOMIC_FLAG)
        for i, (M, N, K) in enumerate([(37, 45, 2048), (257, 529, 2064), (1, 300, 4096)]):
            p = b.gemm_plan(I8, M, N, K, K, K, N, 1 << 40, 2 << 40, 3 << 40, trans_b=True)
            assert p["split_k"] > 1 and p["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC_FLAG, p
            A, Bt = _inputs_bt(I8, M, N, K, seed=450 + i + split)
            for pad_c in (0, (-N) % 4 + 4):
                print(f"bt atomic flag config={config} split={split} shape={(M, N, K)} ldc={N + pad_c}", flush=True)
                _check_bt(I8, A, Bt, g.gemm_gpu_bt(I8, A, Bt, pad=(0, 0, pad_c)))


@pytest.mark.parametrize("split,reduce", [(1, -1), (3, 0), (3, 1), (3, 2)], ids=["s1", "s3sep", "s3fused", "s3atomic"])
@pytest.mark.parametrize("config", BT_CONFIGS)
@pytest.mark.parametrize("dtype", [I8, BF], ids=["i8", "bf16"])
def test_every_bt_config_matches_oracle(dtype, config, split, reduce):
    g.force(dtype, b.GEMM_KERNEL_AUTO, config, split, reduce)
    for i, (M, N, K) in enumerate(VEC_SHAPES):
        A, Bt = _inputs_bt(dtype, M, N, K, seed=300 + i)
        print(f"bt dtype={dtype} config={config} split={split} reduce={reduce} shape={(M, N, K)}", flush=True)
        _check_bt(dtype, A, Bt, g.gemm_gpu_bt(dtype, A, Bt))
    for i, (M, N, K) in enumerate(ODD_SHAPES):
        A, Bt = _inputs_bt(dtype, M, N, K, seed=400 + i)
        if config in GENERIC_CONFIGS:
            print(f"bt dtype={dtype} config={config} split={split} odd shape={(M, N, K)}", flush=True)
            _check_bt(dtype, A, Bt, g.gemm_gpu_bt(dtype, A, Bt))
        else:
            dA, lda = g.to_dev(A)
            dB, ldbt = g.to_dev(Bt)
            dC, ldc = g.out_buffer(M, N, dtype)
            assert g.call_bt(dtype, M, N, K, dA, lda, dB, ldbt, dC, ldc) == b.GEMM_ERR_UNSUPPORTED


@pytest.mark.parametrize("config", [0, 1, 8, 9, 10, 11, 12] + list(range(16, 26)) + list(range(28, 41)))
def test_bt_bf16_integer_valued_is_exact(config):
    M, N, K = 200, 264, 4096
    A = inputs.small_int_bf16_matrix(M, K, seed=17)
    Bt = inputs.small_int_bf16_matrix(N, K, seed=18)
    for split in (1, 5):
        g.force(BF, b.GEMM_KERNEL_AUTO, config, split)
        C = g.gemm_gpu_bt(BF, A, Bt)
        ref = oracle.get().gemm_bf16_f64_bt(A, Bt)
        assert np.array_equal(C.astype(np.float64), ref), (config, split)


@pytest.mark.parametrize("dtype", [I8, BF], ids=["i8", "bf16"])
@pytest.mark.parametrize("pad", [(16, 16, 16), (0, 48, 0), (3, 5, 7)])
def test_bt_strides_and_canaries(dtype, pad):
    M, N, K = 150, 136, 272
    A, Bt = _inputs_bt(dtype, M, N, K, seed=5)
    dA, lda = g.to_dev(A, pad[0])
    dB, ldbt = g.to_dev(Bt, pad[1])
    sentinel = -99 if dtype == I8 else -0.25
    dC, ldc = g.out_buffer(M, N, dtype, pad[2], sentinel=sentinel)
    assert g.call_bt(dtype, M, N, K, dA, lda, dB, ldbt, dC, ldc) == b.GEMM_OK
    torch.cuda.synchronize()
    host = dC.cpu().numpy()
    C = host[: M * ldc].reshape(M, ldc)
    _check_bt(dtype, A, Bt, np.ascontiguousarray(C[:, :N]))
    assert (C[:, N:] == sentinel).all() and (host[M * ldc:] == sentinel).all()


def _sampled_rows(M, seed=5):
    rng = np.random.default_rng(seed)
    rows = {0, M - 1, M // 2}
    rows.update(int(x) for x in rng.integers(0, M, size=5))
    return sorted(r for r in rows if 0 <= r < M)


BIG = inputs.SQUARE + inputs.RECT + inputs.SKINNY


@pytest.mark.parametrize("dtype,M,K,N", BIG, ids=[f"{c[0]}-{c[1]}x{c[2]}x{c[3]}" for c in BIG])
def test_bt_full_size_workloads(dtype, M, K, N):
    d = I8 if dtype == "int8" else BF
    fake = 1 << 40
    plan = b.gemm_plan(d, M, N, K, K, K, N, fake, 2 * fake, 3 * fake, trans_b=True)
    print(f"bt full-size {dtype} M={M} K={K} N={N} plan={plan['name']} split={plan['split_k']}", flush=True)
    A, Bt = _inputs_bt(d, M, N, K, seed=0)
    C = g.gemm_gpu_bt(d, A, Bt)
    o = oracle.get()
    rows = _sampled_rows(M)
    Ar = np.ascontiguousarray(A[rows])
    if d == I8:
        assert o.freivalds_i8_i32_bt(A, Bt, np.ascontiguousarray(C), trials=2) == 0
        ref, ovf = o.gemm_i8_i32_bt(Ar, Bt)
        assert ovf == 0 and np.array_equal(C[rows], ref)
    else:
        ref = o.gemm_bf16_f64_bt(Ar, Bt)
        amax_a = float(np.max(np.abs(inputs.f32_from_bf16_bits(A))))
        amax_b = float(np.max(np.abs(inputs.f32_from_bf16_bits(Bt))))
        assert oracle.normalized_error(C[rows], ref, K, amax_a, amax_b) <= g.BF16_TOL
        assert np.all(np.isfinite(C))


def test_bt_matches_row_major_bitwise():
    """The column-major and row-major paths compute the same int8 C, and for integer-valued
    bf16 the same exact C, on a full-size square problem."""
    M = N = K = 2048
    A, Bt = _inputs_bt(I8, M, N, K, seed=3)
    c_bt = g.gemm_gpu_bt(I8, A, Bt)
    c_rm = g.gemm_gpu(I8, A, np.ascontiguousarray(Bt.T))
    assert np.array_equal(c_bt, c_rm)


def test_torch_helpers_accept_column_major_b():
    M, N, K = 130, 264, 520
    A, Bt = _inputs_bt(I8, M, N, K, seed=1)
    tA, tW = torch.from_numpy(A).to(g.DEV), torch.from_numpy(Bt).to(g.DEV)
    C = b.mm_i8_i32(tA, tW.t())                      # W.t(): a K x N column-major view
    _check_bt(I8, A, Bt, C.cpu().numpy())
    A, Bt = _inputs_bt(BF, M, N, K, seed=2)
    tA = torch.from_numpy(A.view(np.int16)).to(g.DEV).view(torch.bfloat16)
    tW = torch.from_numpy(Bt.view(np.int16)).to(g.DEV).view(torch.bfloat16)
    C = b.mm_bf16_f32(tA, tW.t())
    _check_bt(BF, A, Bt, C.cpu().numpy())
