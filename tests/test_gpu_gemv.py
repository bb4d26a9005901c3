"""Matrix-vector (M = 1) kernels vs the CPU oracle, both B layouts, through the C ABI
(needs an MI355X).  int8 bit-exact; bf16 within the normalised tolerance and exact on
integer-valued operands."""
import numpy as np
import pytest

from oracle import oracle
from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import inputs
import gpu_helpers as g

pytestmark = pytest.mark.gpu
I8, BF = g.I8, g.BF
GEMV_RM, GEMV_BT = 26, 27


@pytest.fixture(autouse=True)
def _reset_plan():
    g.unforce()
    yield
    g.unforce()


def _name(dtype):
    return "int8" if dtype == I8 else "bf16"


def _check_bt(dtype, A, Bt, C):
    o = oracle.get()
    if dtype == I8:
        ref, ovf = o.gemm_i8_i32_bt(A, Bt)
        assert ovf == 0
        assert np.array_equal(C, ref), np.argwhere(C != ref)[:3].tolist()
    else:
        err = g.bf16_error(A, np.ascontiguousarray(Bt.T), C, o.gemm_bf16_f64_bt(A, Bt))
        assert err <= g.BF16_TOL, err


# N ragged against the 1024-column (row-major) and 16-column (column-major) blocks;
# K from one 16-byte piece to several slices.
SHAPES = [(16, 16), (48, 272), (1040, 1040), (2064, 4096), (4112, 528), (14336, 4096), (4096, 14336)]
SPLITS = [(1, -1), (3, 0), (3, 1), (7, 1), (5, 2), (5, 3), (32, 3)]
SPLIT_IDS = ["s1", "s3sep", "s3fused", "s7fused", "s5atomic", "s5flag", "s32flag"]


@pytest.mark.parametrize("split,reduce", SPLITS, ids=SPLIT_IDS)
@pytest.mark.parametrize("dtype", [I8, BF], ids=["i8", "bf16"])
def test_gemv_row_major_b(dtype, split, reduce):
    g.force(dtype, b.GEMM_KERNEL_AUTO, GEMV_RM, split, reduce)
    for i, (N, K) in enumerate(SHAPES):
        A, B = inputs.make_inputs(_name(dtype), 1, N, K, seed=500 + i)
        print(f"gemv dtype={dtype} split={split} reduce={reduce} N={N} K={K}", flush=True)
        (g.check_i8 if dtype == I8 else g.check_bf16)(A, B, g.gemm_gpu(dtype, A, B))


@pytest.mark.parametrize("split,reduce", SPLITS, ids=SPLIT_IDS)
@pytest.mark.parametrize("dtype", [I8, BF], ids=["i8", "bf16"])
def test_gemv_column_major_b(dtype, split, reduce):
    g.force(dtype, b.GEMM_KERNEL_AUTO, GEMV_BT, split, reduce)
    for i, (N, K) in enumerate(SHAPES):
        A, B = inputs.make_inputs(_name(dtype), 1, N, K, seed=600 + i)
        Bt = np.ascontiguousarray(B.T)
        print(f"gemv_bt dtype={dtype} split={split} reduce={reduce} N={N} K={K}", flush=True)
        _check_bt(dtype, A, Bt, g.gemm_gpu_bt(dtype, A, Bt))


@pytest.mark.parametrize("config", [GEMV_RM, GEMV_BT])
def test_gemv_bf16_integer_valued_is_exact(config):
    N, K = 2064, 4096
    A = inputs.small_int_bf16_matrix(1, K, seed=27)
    B = inputs.small_int_bf16_matrix(K, N, seed=28)
    ref = oracle.get().gemm_bf16_f64(A, B)
    for split in (1, 5):
        g.force(BF, b.GEMM_KERNEL_AUTO, config, split)
        C = g.gemm_gpu(BF, A, B) if config == GEMV_RM else g.gemm_gpu_bt(BF, A, np.ascontiguousarray(B.T))
        assert np.array_equal(C.astype(np.float64), ref), (config, split)


@pytest.mark.parametrize("config", [GEMV_RM, GEMV_BT])
def test_gemv_int8_extremes(config):
    """(-128)(-128) over K = 14336 = 234,881,024, the largest sum of the workload sweep."""
    N, K = 1040, 14336
    A = np.full((1, K), -128, np.int8)
    B = np.full((K, N), -128, np.int8)
    B[:, 1::3] = 127
    for split in (1, 4):
        g.force(I8, b.GEMM_KERNEL_AUTO, config, split)
        C = g.gemm_gpu(I8, A, B) if config == GEMV_RM else g.gemm_gpu_bt(I8, A, np.ascontiguousarray(B.T))
        expect = np.where(np.arange(N) % 3 == 1, -16256 * K, 16384 * K)
        assert np.array_equal(C[0], expect), split


def test_gemv_padded_strides_and_canaries():
    """Row strides beyond the widths; nothing past C's row is written."""
    N, K = 1040, 528
    A, B = inputs.make_inputs("int8", 1, N, K, seed=9)
    g.force(I8, b.GEMM_KERNEL_AUTO, GEMV_RM, 3, 1)
    C = g.gemm_gpu(I8, A, B, pad=(16, 32, 48))
    g.check_i8(A, B, C)
    dA, lda = g.to_dev(A)
    dB, ldb = g.to_dev(B)
    dC, ldc = g.out_buffer(1, N, I8, pad_cols=64)
    assert g.call(I8, 1, N, K, dA, lda, dB, ldb, dC, ldc) == b.GEMM_OK
    host = dC.cpu().numpy()
    assert (host[N:] == -123456789).all()


@pytest.mark.parametrize("dtype,M,K,N", [c for c in inputs.SKINNY if c[1] == 1],
                         ids=[f"{c[0]}-{c[2]}x{c[3]}" for c in inputs.SKINNY if c[1] == 1])
def test_full_size_m1_selector_plan(dtype, M, K, N):
    """The full-size M = 1 workloads (B row-major) through the selector's plan, whichever kernel
    it picks (the row-major GEMV kernel for int8, a ring plan for bf16, as measured), against
    the whole oracle row."""
    d = I8 if dtype == "int8" else BF
    fake = 1 << 40
    plan = b.gemm_plan(d, M, N, K, K, N, N, fake, 2 * fake, 3 * fake)
    print(f"full-size {dtype} M=1 K={K} N={N} plan={plan['name']} split={plan['split_k']}", flush=True)
    A, B = inputs.make_inputs(dtype, M, N, K, seed=0)
    (g.check_i8 if d == I8 else g.check_bf16)(A, B, g.gemm_gpu(d, A, B))
