"""Reduced-precision outputs (int8 -> int8 / int16 with a power-of-two requantisation,
bf16 -> bf16) vs the oracle, through the C ABI (needs an MI355X).

int8 outputs must equal the oracle's requantisation of the exact int32 results
bit for bit.  bf16 outputs round the kernel's fp32 sum, the oracle rounds the exact
sum: they must agree to within one bf16 step (a rounding boundary can fall between
the two sums), stay within half a bf16 step plus the fp32 calls' normalised bound
of the exact sum, and agree exactly on integer-valued operands, where the fp32 sum
is exact."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import inputs
import gpu_helpers as g

pytestmark = pytest.mark.gpu
I8, BF = g.I8, g.BF
# One or two configurations of every kernel family; GEMV (26 row-major, 27 column-major) for M = 1.
CONFIGS = [0, 2, 6, 8, 10, 13, 14, 16, 20]
BT_CONFIGS = [0, 10, 16, 20]
SHAPES = [(300, 272, 1040), (64, 256, 128), (1, 48, 528)]
I8_EPILOGUES = [("i8", 0), ("i8", 6), ("i8", 12), ("i8", 17), ("i16", 0), ("i16", 9), ("i16", 14)]
SENTINEL = {"i8": -77, "i16": -7777, "bf16": 0x7FC1}


@pytest.fixture(autouse=True)
def _reset_plan():
    g.unforce()
    yield
    g.unforce()


def run_epilogue(kind, A, B, shift=0, bt=False, pad=8):
    """Runs gemm_i8_i8 / gemm_i8_i16 / gemm_bf16_bf16 (or the *_bt form, B then being Bt)
    and returns C (M x N) as numpy; checks nothing past each row's N outputs was written."""
    M, K = A.shape
    N = B.shape[0] if bt else B.shape[1]
    dA, lda = g.to_dev(A)
    dB, ldb = g.to_dev(B)
    ldc = N + pad
    tdt = {"i8": torch.int8, "i16": torch.int16, "bf16": torch.int16}[kind]
    fill = SENTINEL[kind] if kind != "bf16" else np.int16(np.uint16(SENTINEL[kind]).view(np.int16))
    buf = torch.full((M * ldc + 64,), int(fill), dtype=tdt, device=g.DEV)
    st = torch.cuda.current_stream().cuda_stream
    name = {"i8": "gemm_i8_i8", "i16": "gemm_i8_i16", "bf16": "gemm_bf16_bf16"}[kind] + ("_bt" if bt else "")
    fn = getattr(b, name)
    args = (M, N, K, dA.data_ptr(), max(lda, 1), dB.data_ptr(), max(ldb, 1), buf.data_ptr(), ldc)
    rc = fn(*args, shift, st) if kind != "bf16" else fn(*args, st)
    assert rc == b.GEMM_OK, b.gemm_status_string(rc)
    torch.cuda.synchronize()
    host = buf.cpu().numpy()
    full = host[: M * ldc].reshape(M, ldc)
    assert (full[:, N:] == fill).all() and (host[M * ldc:] == fill).all(), "wrote outside C"
    C = full[:, :N]
    return C.view(np.uint16) if kind == "bf16" else C


def _bf16_value(bits):
    return inputs.f32_from_bf16_bits(bits).astype(np.float64)


def check_i8(kind, shift, A, B, C, bt=False):
    o = oracle.get()
    exact, ovf = o.gemm_i8_i32_bt(A, B) if bt else o.gemm_i8_i32(A, B)
    assert ovf == 0
    ref = o.requant_i32(exact, shift, 8 if kind == "i8" else 16)
    bad = np.argwhere(C != ref)
    assert bad.size == 0, f"{len(bad)} mismatches, first {bad[:3].tolist()}"


def check_bf16(A, B, C, bt=False):
    o = oracle.get()
    exact = o.gemm_bf16_f64_bt(A, B) if bt else o.gemm_bf16_f64(A, B)
    ref_bits = o.round_bf16(exact)
    got, ref = _bf16_value(C), _bf16_value(ref_bits)
    # one bf16 step at the reference's magnitude (8 significant bits)
    mag = np.maximum(np.abs(ref), 2.0 ** -126)
    step = 2.0 ** (np.floor(np.log2(mag)) - 7)
    assert np.all(np.abs(got - ref) <= step), np.argwhere(np.abs(got - ref) > step)[:3].tolist()
    # and against the exact sum: half a bf16 step of output rounding on top of the fp32
    # path's own bound (the normalised bar of the fp32-output calls)
    Bn = np.ascontiguousarray(B.T) if bt else B
    amax_a = float(np.max(np.abs(_bf16_value(A))))
    amax_b = float(np.max(np.abs(_bf16_value(Bn))))
    bound = 2.0 ** -8 * np.abs(exact) + g.BF16_TOL * A.shape[1] * amax_a * amax_b
    assert np.all(np.abs(got - exact) <= bound)


@pytest.mark.parametrize("split,reduce", [(1, -1), (3, 0), (3, 1), (3, 2), (3, 3)],
                         ids=["s1", "s3sep", "s3fused", "s3atomic", "s3flag"])
@pytest.mark.parametrize("config", CONFIGS)
def test_reduced_outputs_every_family(config, split, reduce):
    for i, (M, N, K) in enumerate(SHAPES):
        for kind, shift in I8_EPILOGUES:
            g.force(I8, b.GEMM_KERNEL_AUTO, config, split, reduce)
            A, B = inputs.make_inputs("int8", M, N, K, seed=700 + i)
            print(f"epilogue {kind} shift={shift} config={config} split={split} shape={(M, N, K)}", flush=True)
            check_i8(kind, shift, A, B, run_epilogue(kind, A, B, shift))
        g.force(BF, b.GEMM_KERNEL_AUTO, config, split, reduce)
        A, B = inputs.make_inputs("bf16", M, N, K, seed=800 + i)
        print(f"epilogue bf16 config={config} split={split} shape={(M, N, K)}", flush=True)
        check_bf16(A, B, run_epilogue("bf16", A, B))


@pytest.mark.parametrize("split,reduce", [(1, -1), (3, 1)], ids=["s1", "s3fused"])
@pytest.mark.parametrize("config", BT_CONFIGS)
def test_reduced_outputs_column_major_b(config, split, reduce):
    for i, (M, N, K) in enumerate(SHAPES):
        for kind, shift in I8_EPILOGUES[::2]:
            g.force(I8, b.GEMM_KERNEL_AUTO, config, split, reduce)
            A, B = inputs.make_inputs("int8", M, N, K, seed=900 + i)
            Bt = np.ascontiguousarray(B.T)
            print(f"epilogue bt {kind} shift={shift} config={config} split={split} shape={(M, N, K)}", flush=True)
            check_i8(kind, shift, A, Bt, run_epilogue(kind, A, Bt, shift, bt=True), bt=True)
        g.force(BF, b.GEMM_KERNEL_AUTO, config, split, reduce)
        A, B = inputs.make_inputs("bf16", M, N, K, seed=950 + i)
        Bt = np.ascontiguousarray(B.T)
        check_bf16(A, Bt, run_epilogue("bf16", A, Bt, bt=True), bt=True)


@pytest.mark.parametrize("config,bt", [(26, False), (27, True)], ids=["gemv", "gemv_bt"])
def test_reduced_outputs_gemv(config, bt):
    M, N, K = 1, 2064, 4096
    for split in (1, 4):
        for kind, shift in I8_EPILOGUES:
            g.force(I8, b.GEMM_KERNEL_AUTO, config, split, 1)
            A, B = inputs.make_inputs("int8", M, N, K, seed=1000 + split)
            Bx = np.ascontiguousarray(B.T) if bt else B
            check_i8(kind, shift, A, Bx, run_epilogue(kind, A, Bx, shift, bt=bt), bt=bt)
        g.force(BF, b.GEMM_KERNEL_AUTO, config, split, 1)
        A, B = inputs.make_inputs("bf16", M, N, K, seed=1100 + split)
        Bx = np.ascontiguousarray(B.T) if bt else B
        check_bf16(A, Bx, run_epilogue("bf16", A, Bx, bt=bt), bt=bt)


@pytest.mark.parametrize("config", [0, 10, 16, 20])
def test_bf16_to_bf16_exact_on_integer_operands(config):
    """Integer-valued operands: the fp32 sum is exact, so its bf16 rounding is unique."""
    M, N, K = 200, 264, 4096
    A = inputs.small_int_bf16_matrix(M, K, seed=41)
    B = inputs.small_int_bf16_matrix(K, N, seed=42)
    ref = oracle.get().round_bf16(oracle.get().gemm_bf16_f64(A, B))
    for split in (1, 5):
        g.force(BF, b.GEMM_KERNEL_AUTO, config, split)
        assert np.array_equal(run_epilogue("bf16", A, B), ref), (config, split)


def test_int8_saturation_and_ties():
    """Results at exact halves and far outside the output ranges."""
    M, N, K = 64, 256, 2048
    A = np.full((M, K), -128, np.int8)
    B = np.ones((K, N), np.int8)
    B[:, 1::2] = -1
    # exact results: -262144 (even columns), +262144 (odd columns) = +-2^18
    for kind, shift, lo_hi in (("i8", 0, (-128, 127)), ("i16", 0, (-32768, 32767)), ("i8", 11, (-128, 127)),
                               ("i16", 3, (-32768, 32767)), ("i16", 4, (-16384, 16384)), ("i8", 12, (-64, 64))):
        for split in (1, 4):
            g.force(I8, b.GEMM_KERNEL_AUTO, 10, split)
            C = run_epilogue(kind, A, B, shift)
            assert (C[:, 0::2] == lo_hi[0]).all() and (C[:, 1::2] == lo_hi[1]).all(), (kind, shift, split)
    # ties: sums of 3 over shift 1 -> 1.5 -> 2; sums of 5 -> 2.5 -> 2; -3 -> -1.5 -> -2
    A = np.ones((M, K), np.int8)
    B = np.zeros((K, N), np.int8)
    B[:3, 0::4] = 1
    B[:5, 1::4] = 1
    B[:3, 2::4] = -1
    B[:7, 3::4] = 1
    C = run_epilogue("i8", A, B, 1)
    assert (C[:, 0::4] == 2).all() and (C[:, 1::4] == 2).all() and (C[:, 2::4] == -2).all() and (C[:, 3::4] == 4).all()


@pytest.mark.parametrize("dtype", ["int8", "bf16"])
def test_full_size_8192_reduced_outputs(dtype):
    """The headline size through the selector's plan: sampled rows against the oracle."""
    S = 8192
    A, B = inputs.make_inputs(dtype, S, S, S, seed=0)
    rows = sorted({0, 1, S // 2, S - 1, 1234, 5678})
    o = oracle.get()
    if dtype == "int8":
        for kind, shift in (("i8", 14), ("i16", 6)):
            C = run_epilogue(kind, A, B, shift, pad=0)
            exact, ovf = o.gemm_i8_i32(np.ascontiguousarray(A[rows]), B)
            assert ovf == 0
            assert np.array_equal(C[rows], o.requant_i32(exact, shift, 8 if kind == "i8" else 16))
    else:
        C = run_epilogue("bf16", A, B, pad=0)
        check_bf16(np.ascontiguousarray(A[rows]), B, np.ascontiguousarray(C[rows]))


@pytest.mark.parametrize("cfg", [0, 10, 16, 20])
def test_bf16_infinities_and_nans_propagate(cfg):
    """Infinite and NaN operands: every output is NaN, +inf, -inf or finite exactly where the
    oracle's exact sum is (IEEE sums of the same products; the class of such a sum does not
    depend on the summation order while the finite part cannot overflow, as here), through the
    fp32 output and the bf16 output, whose rounding must keep a NaN a NaN."""
    rng = np.random.default_rng(40 + cfg)
    M, K, N = 64, 96, 80
    a = rng.integers(-4, 5, size=(M, K)).astype(np.float32)
    bvals = np.array([-4, -3, -2, -1, 1, 2, 3, 4], dtype=np.float32)
    bmat = bvals[rng.integers(0, 8, size=(K, N))]
    a[3, 5] = np.inf
    a[7, 1] = -np.inf
    a[11, 9] = np.nan
    a[13, 2], a[13, 40] = np.inf, -np.inf      # +inf and -inf products meet: NaN or inf by sign
    a[20, 0] = np.inf
    bmat[0, 17] = 0.0                          # inf * 0 = NaN in one column of row 20
    A, B = inputs.bf16_bits_from_f32(a), inputs.bf16_bits_from_f32(bmat)
    ref = oracle.get().gemm_bf16_f64(A, B)
    g.force(BF, b.GEMM_KERNEL_AUTO, cfg)
    C = g.gemm_gpu(BF, A, B).astype(np.float64)
    assert np.array_equal(np.isnan(C), np.isnan(ref)), "NaN positions differ"
    fin = np.isfinite(ref)
    assert np.array_equal(C[~np.isnan(ref) & ~fin], ref[~np.isnan(ref) & ~fin]), "infinities differ"
    assert np.array_equal(C[fin], ref[fin]), "finite (integer-valued) outputs differ"
    assert np.isnan(ref).any() and (np.isinf(ref) & (ref > 0)).any() and (np.isinf(ref) & (ref < 0)).any()
    Cb = run_epilogue("bf16", A, B)
    nan_b = ((Cb & 0x7F80) == 0x7F80) & ((Cb & 0x007F) != 0)
    assert np.array_equal(nan_b, np.isnan(ref)), "bf16 NaN positions differ"
    ref_bits = oracle.get().round_bf16(ref)
    assert np.array_equal(Cb[~np.isnan(ref)], ref_bits[~np.isnan(ref)]), "bf16 non-NaN outputs differ"
