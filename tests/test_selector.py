"""The shape-driven selector (pure host code, exercised through gemm_plan)."""
import itertools
import math

import pytest

from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import inputs

I8, BF = b.GEMM_DTYPE_I8_I32, b.GEMM_DTYPE_BF16_F32
DT = {"int8": I8, "bf16": BF}
ESZ = {I8: 1, BF: 2}
AL = 1 << 40    # 16-byte aligned fake addresses, far apart (never dereferenced)
LDS_MAX = 160 * 1024


def plan(dtype, M, N, K, lda=None, ldb=None, ldc=None, off=0):
    return b.gemm_plan(dtype, M, N, K, lda or max(K, 1), ldb or max(N, 1), ldc or max(N, 1),
                       AL + off, 2 * AL, 3 * AL)


def check_invariants(p, dtype, M, N, K):
    stage = 128 // ESZ[dtype]
    assert p["lds_bytes"] <= LDS_MAX
    assert p["bk"] == stage
    tiles_m = -(-M // p["bm"])
    tiles_n = -(-N // p["bn"])
    assert p["grid"] == tiles_m * tiles_n * p["split_k"]
    if K > 0:
        assert p["k_chunk"] % stage == 0 and p["k_chunk"] > 0
        assert p["split_k"] * p["k_chunk"] >= K > (p["split_k"] - 1) * p["k_chunk"]
    else:
        assert p["split_k"] == 1
    atomic = p["reduce_in_kernel"] in (b.GEMM_REDUCE_ATOMIC, b.GEMM_REDUCE_ATOMIC_FLAG)
    planes = p["split_k"] > 1 and not atomic
    assert p["workspace_bytes"] == (p["split_k"] * M * N * 4 if planes else 0)
    if atomic:
        assert dtype == I8 and p["split_k"] > 1
    if p["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC_FLAG:
        assert p["kernel"] in (b.GEMM_KERNEL_RING, b.GEMM_KERNEL_GEMV)
    assert p["grid"] < 2 ** 31


SIZES = [1, 2, 3, 15, 16, 17, 31, 33, 63, 64, 65, 127, 129, 255, 257, 1000, 4096]


@pytest.mark.parametrize("dtype", [I8, BF])
def test_every_shape_gets_a_valid_plan(dtype):
    for M, N, K in itertools.product([1, 17, 64, 257, 4096], [1, 8, 33, 256, 4000], [0, 1, 16, 100, 8192]):
        p = plan(dtype, M, N, K)
        check_invariants(p, dtype, M, N, K)


@pytest.mark.parametrize("dtype", [I8, BF])
def test_alignment_routes_to_generic(dtype):
    # K not a multiple of the 16-byte chunk -> element-wise loaders
    p = plan(dtype, 512, 512, 4096 + 1)
    assert p["kernel"] == b.GEMM_KERNEL_GENERIC
    # misaligned A pointer -> generic
    p = plan(dtype, 512, 512, 4096, off=ESZ[dtype])
    assert p["kernel"] == b.GEMM_KERNEL_GENERIC
    # N not a multiple of 8 -> generic
    p = plan(dtype, 512, 4100, 4096)
    assert p["kernel"] == b.GEMM_KERNEL_GENERIC
    # everything aligned -> vectorised family
    p = plan(dtype, 512, 512, 4096)
    assert p["kernel"] in (b.GEMM_KERNEL_MACRO, b.GEMM_KERNEL_SKINNY, b.GEMM_KERNEL_DIRECT, b.GEMM_KERNEL_RING)


@pytest.mark.parametrize("dtype", ["int8", "bf16"])
def test_workload_plans(dtype):
    d = DT[dtype]
    big = plan(d, 8192, 8192, 8192)
    # the square 8192 problem fills the chip with large tiles (256 x 256, or two 128 x 256
    # workgroups per compute unit) and needs no split
    assert big["bm"] * big["bn"] >= 128 * 256 and big["bn"] == 256 and big["split_k"] == 1
    assert big["grid"] >= 4 * 256
    for (_, M, K, N) in [c for c in inputs.ALL_CONFIGS if c[0] == dtype]:
        p = plan(d, M, N, K)
        check_invariants(p, d, M, N, K)
        assert p["kernel"] != b.GEMM_KERNEL_GENERIC


def test_skinny_shapes_split_k():
    # 16 rows, 4096 columns: 16 N tiles alone would leave most CUs idle
    for d in (I8, BF):
        p = plan(d, 16, 4096, 14336)
        assert p["split_k"] > 1 and p["grid"] >= 64


def test_forced_plans():
    try:
        assert b.gemm_force_plan(I8, b.GEMM_KERNEL_GENERIC, -1, 3) == b.GEMM_OK
        p = plan(I8, 300, 200, 1000)
        assert p["kernel"] == b.GEMM_KERNEL_GENERIC and p["split_k"] == 3
        assert b.gemm_force_plan(I8, b.GEMM_KERNEL_MACRO, 2, 1) == b.GEMM_OK
        p = plan(I8, 300, 256, 1024)
        assert p["config"] == 2 and p["split_k"] == 1
        # a forced vectorised plan cannot run misaligned K
        with pytest.raises(b.GemmError) as e:
            plan(I8, 300, 256, 1001)
        assert e.value.status == b.GEMM_ERR_UNSUPPORTED
        # split larger than the number of stages is clamped
        assert b.gemm_force_plan(BF, b.GEMM_KERNEL_AUTO, -1, 64) == b.GEMM_OK
        p = plan(BF, 64, 64, 128)
        assert p["split_k"] == 2
    finally:
        b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, -1, 0)
        b.gemm_force_plan(BF, b.GEMM_KERNEL_AUTO, -1, 0)


def test_traffic_model_follows_eqs_6_to_8():
    # A reads scale with the number of N tiles, B reads with the number of M tiles (Eqs. 6-7),
    # C is written once (Eq. 8); no split -> no partial traffic.
    M = N = K = 8192
    p = plan(I8, M, N, K)
    tiles_m, tiles_n = M // p["bm"], N // p["bn"]
    expect = M * K * tiles_n + K * N * tiles_m + M * N * 4
    assert abs(p["model_traffic_bytes"] - expect) < 1e-6 * expect


def test_plans_are_deterministic():
    a = plan(BF, 2048, 11008, 4096)
    c = plan(BF, 2048, 11008, 4096)
    assert a == c


def _tuned_entries():
    import os
    import re
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                        "paper_2512_13282_amd", "csrc", "tuned_plans.inc")
    out = []
    for line in open(path):
        m = re.match(r"\s*\{(-?\d+), (\d+), (\d+), (\d+), (\d+), (\d+), (-?\d+), ([01])\},", line)
        if m:
            out.append(tuple(int(x) for x in m.groups()))
    return out


def test_tuned_plans_are_valid_and_used():
    """Every measured plan names a vectorised configuration that can run its shape, and
    gemm_plan returns it (no override active, aligned operands)."""
    entries = _tuned_entries()
    assert entries, "tuned_plans.inc holds no plans"
    for (d, M, N, K, cfg, split, reduce, bt) in entries:
        p = plan_bt(d, M, N, K) if bt else plan(d, M, N, K)
        assert p["config"] == cfg, (d, M, N, K, p["name"])
        if reduce >= 0 and p["split_k"] > 1:
            assert p["reduce_in_kernel"] == reduce
        assert p["kernel"] != b.GEMM_KERNEL_GENERIC
        check_invariants(p, d, M, N, K)


def test_shapes_borrow_the_nearest_tuned_plan():
    """M <= 2048 without a plan of its own, at a (dtype, B layout, N, K) that has tuned plans:
    the configuration and split of the tuned plan with the nearest M on a log scale (the
    larger M on a tie) among those whose tile covers as many tile rows at both sizes."""
    groups = {}
    for (d, M, N, K, cfg, split, reduce, bt) in _tuned_entries():
        if M <= 2048:
            groups.setdefault((d, bt, N, K), {})[M] = (cfg, split)
    checked = 0
    for (d, bt, N, K), by_m in groups.items():
        pl = plan_bt if bt else plan
        bm = {m: pl(d, m, N, K)["bm"] for m in by_m}
        for M in list(range(1, 257)) + list(range(260, 2049, 4)):
            if M in by_m:
                continue
            p = pl(d, M, N, K)
            check_invariants(p, d, M, N, K)
            same_rows = [m for m in by_m if -(-m // bm[m]) == -(-M // bm[m])]
            if not same_rows:
                continue
            near = min(same_rows, key=lambda m: (abs(math.log(m / M)), -m))
            assert (p["config"], p["split_k"]) == by_m[near], (d, bt, M, N, K, p["name"], near)
            checked += 1
    assert checked >= 10000


def test_tuned_table_is_the_tuner_default_list():
    """The compiled table holds one measured plan for every shape of the tuner's default
    list and nothing else, so re-running the tuner with no arguments reproduces it."""
    from paper_2512_13282_amd import tune
    shapes, warm = tune.default_shapes()
    want = {(DT[s[0]], s[1], s[3], s[2], int(len(s) > 4)) for s in shapes}
    have = [(d, M, N, K, bt) for (d, M, N, K, cfg, split, reduce, bt) in _tuned_entries()]
    assert len(have) == len(set(have)), "a shape appears twice"
    assert set(have) == want
    assert all((s[0], s[1], s[2], s[3]) in inputs.ALL_CONFIGS for s in warm)


def test_tuned_plans_skip_misaligned_operands():
    # the same shape with a misaligned A pointer falls back to the alignment-agnostic family
    (d, M, N, K, cfg, split, reduce, bt) = _tuned_entries()[0]
    p = plan(d, M, N, K, off=ESZ[d])
    assert p["kernel"] == b.GEMM_KERNEL_GENERIC


def test_split_k_reduction_choice():
    """bf16: a small per-tile reduction (one row of output) is summed in the GEMM kernel by the
    last slice, a large one (many rows times many slices) by the separate kernel.  int8: an
    atomic reduction, whatever the size: C zeroed by each tile's first slice on ring and GEMV
    kernels, by a fill kernel on the others.  Forcing a reduction is reflected in the plan, and
    split_k == 1 reports none."""
    try:
        for d in (I8, BF):
            assert b.gemm_force_plan(d, b.GEMM_KERNEL_AUTO, 14, 16) == b.GEMM_OK
        small = plan(BF, 1, 4096, 14336)
        assert small["split_k"] == 16 and small["reduce_in_kernel"] == b.GEMM_REDUCE_LAST_SLICE
        assert plan(I8, 1, 4096, 14336)["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC
        for d in (I8, BF):
            assert b.gemm_force_plan(d, b.GEMM_KERNEL_AUTO, 3, 32) == b.GEMM_OK
        large = plan(BF, 128, 4096, 16384)
        assert large["split_k"] == 32 and large["reduce_in_kernel"] == b.GEMM_REDUCE_SEPARATE
        assert plan(I8, 128, 4096, 16384)["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC
        for mode in (b.GEMM_REDUCE_SEPARATE, b.GEMM_REDUCE_LAST_SLICE, b.GEMM_REDUCE_ATOMIC):
            assert b.gemm_force_reduce(I8, mode) == b.GEMM_OK
            assert plan(I8, 128, 4096, 16384)["reduce_in_kernel"] == mode
        assert b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, 3, 1) == b.GEMM_OK
        assert plan(I8, 128, 4096, 16384)["reduce_in_kernel"] == 0
        b.gemm_force_reduce(I8, -1)
        assert b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, 28, 4) == b.GEMM_OK      # ring_32x256_w4_r4
        assert plan(I8, 16, 14336, 4096)["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC_FLAG
        assert b.gemm_force_plan(I8, b.GEMM_KERNEL_GEMV, 26, 8) == b.GEMM_OK      # gemv_1024
        assert plan(I8, 1, 14336, 4096)["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC_FLAG
        assert b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, 14, 4) == b.GEMM_OK      # stream_32x256_s4
        assert plan(I8, 16, 14336, 4096)["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC
    finally:
        for d in (I8, BF):
            b.gemm_force_plan(d, b.GEMM_KERNEL_AUTO, -1, 0)
            b.gemm_force_reduce(d, -1)


def test_atomic_reduction_plans():
    """The atomic split-K reductions are int8-only and need no partial planes; asked of bf16,
    the plan takes the separate reduction instead.  The one whose C is zeroed by the first
    slice runs on ring and GEMV kernels; another family asked for it keeps the fill kernel."""
    try:
        for d in (I8, BF):
            assert b.gemm_force_plan(d, b.GEMM_KERNEL_AUTO, 28, 4) == b.GEMM_OK
            assert b.gemm_force_reduce(d, b.GEMM_REDUCE_ATOMIC) == b.GEMM_OK
        p = plan(I8, 16, 14336, 4096)
        check_invariants(p, I8, 16, 14336, 4096)
        assert p["split_k"] == 4 and p["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC and p["workspace_bytes"] == 0
        q = plan(BF, 16, 14336, 4096)
        check_invariants(q, BF, 16, 14336, 4096)
        assert q["split_k"] == 4 and q["reduce_in_kernel"] == b.GEMM_REDUCE_SEPARATE
        assert q["workspace_bytes"] == 4 * 16 * 14336 * 4
        # C zeroed by the first slice: ring and GEMV kernels only, others keep the fill kernel
        for d in (I8, BF):
            assert b.gemm_force_reduce(d, b.GEMM_REDUCE_ATOMIC_FLAG) == b.GEMM_OK
        p = plan(I8, 16, 14336, 4096)
        check_invariants(p, I8, 16, 14336, 4096)
        assert p["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC_FLAG and p["workspace_bytes"] == 0
        assert plan(BF, 16, 14336, 4096)["reduce_in_kernel"] == b.GEMM_REDUCE_SEPARATE
        assert b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, 14, 4) == b.GEMM_OK      # stream_32x256_s4
        p = plan(I8, 16, 14336, 4096)
        check_invariants(p, I8, 16, 14336, 4096)
        assert p["kernel"] == b.GEMM_KERNEL_SKINNY and p["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC
        assert b.gemm_force_plan(I8, b.GEMM_KERNEL_GEMV, 26, 8) == b.GEMM_OK      # gemv_1024
        p = plan(I8, 1, 14336, 4096)
        check_invariants(p, I8, 1, 14336, 4096)
        assert p["reduce_in_kernel"] == b.GEMM_REDUCE_ATOMIC_FLAG
    finally:
        for d in (I8, BF):
            b.gemm_force_plan(d, b.GEMM_KERNEL_AUTO, -1, 0)
            b.gemm_force_reduce(d, -1)


def plan_bt(dtype, M, N, K, ldbt=None, off=0):
    return b.gemm_plan(dtype, M, N, K, max(K, 1), ldbt or max(K, 1), max(N, 1), AL + off, 2 * AL, 3 * AL,
                       trans_b=True)


@pytest.mark.parametrize("dtype", [I8, BF])
def test_column_major_b_plans(dtype):
    """B stored N x K runs on the configurations built for it (the generic, direct and
    ring families), with the same tiling invariants; alignment of Bt rows is judged on K."""
    for M, N, K in itertools.product([1, 17, 64, 257, 4096], [1, 8, 33, 256, 4000], [0, 1, 16, 100, 8192]):
        p = plan_bt(dtype, M, N, K)
        check_invariants(p, dtype, M, N, K)
        fams = (b.GEMM_KERNEL_GENERIC, b.GEMM_KERNEL_DIRECT, b.GEMM_KERNEL_RING)
        assert p["kernel"] in fams + ((b.GEMM_KERNEL_GEMV,) if M == 1 else ())
        assert p["name"] != "gemv_1024" and not p["name"].startswith("pingpong")
    # N need not be a multiple of 16 bytes for column-major B, K must
    assert plan_bt(dtype, 512, 4100, 4096)["kernel"] in (b.GEMM_KERNEL_DIRECT, b.GEMM_KERNEL_RING)
    assert plan_bt(dtype, 512, 512, 4097)["kernel"] == b.GEMM_KERNEL_GENERIC
    assert plan_bt(dtype, 512, 512, 4096, off=ESZ[dtype])["kernel"] == b.GEMM_KERNEL_GENERIC
    big = plan_bt(dtype, 8192, 8192, 8192)
    assert big["kernel"] in (b.GEMM_KERNEL_DIRECT, b.GEMM_KERNEL_RING) and big["bm"] == 256 and big["bn"] == 256


def test_column_major_b_rejects_configs_without_it():
    try:
        for cfg in (2, 6, 13, 14):
            assert b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, cfg, 1) == b.GEMM_OK
            with pytest.raises(b.GemmError) as e:
                plan_bt(I8, 512, 512, 4096)
            assert e.value.status == b.GEMM_ERR_UNSUPPORTED
            plan(I8, 512, 512, 4096)      # the row-major form still runs it
    finally:
        b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, -1, 0)


GEMV_RM, GEMV_BT = 26, 27


@pytest.mark.parametrize("dtype", [I8, BF])
def test_gemv_configs_only_for_one_row(dtype):
    """The matrix-vector kernels run M = 1 only, each with its own B layout."""
    try:
        b.gemm_force_plan(dtype, b.GEMM_KERNEL_AUTO, GEMV_RM, 0)
        p = plan(dtype, 1, 14336, 4096)
        assert p["name"] == "gemv_1024" and p["kernel"] == b.GEMM_KERNEL_GEMV
        assert p["mfma_m"] == p["mfma_n"] == p["mfma_k"] == 0 and p["bm"] == 1
        check_invariants(p, dtype, 1, 14336, 4096)
        for M in (2, 16):
            with pytest.raises(b.GemmError) as e:
                plan(dtype, M, 14336, 4096)
            assert e.value.status == b.GEMM_ERR_UNSUPPORTED
        with pytest.raises(b.GemmError):
            plan_bt(dtype, 1, 14336, 4096)                  # row-major-B kernel only
        b.gemm_force_plan(dtype, b.GEMM_KERNEL_AUTO, GEMV_BT, 0)
        p = plan_bt(dtype, 1, 4096, 14336)
        assert p["name"] == "gemv_bt_16" and p["bn"] == 16
        check_invariants(p, dtype, 1, 4096, 14336)
        with pytest.raises(b.GemmError):
            plan(dtype, 1, 4096, 14336)                     # column-major-B kernel only
    finally:
        b.gemm_force_plan(dtype, b.GEMM_KERNEL_AUTO, -1, 0)


@pytest.mark.parametrize("dtype", [I8, BF])
def test_memory_bound_ties_go_to_the_faster_kernel(dtype):
    # (M, K, N) = (2048, 256, 8192): every 256 x 256 config moves the same bytes, so the
    # modelled totals tie; the choice must be the tied plan with the shortest compute time.
    M, K, N = 2048, 256, 8192
    p = plan(dtype, M, N, K)
    assert p["model_t_mem_us"] > p["model_t_comp_us"]
    try:
        for cfg in range(64):
            if b.gemm_force_plan(dtype, b.GEMM_KERNEL_AUTO, cfg, 0) != b.GEMM_OK:
                break
            try:
                q = plan(dtype, M, N, K)
            except b.GemmError:
                continue
            same_total = (abs(max(q["model_t_comp_us"], q["model_t_mem_us"]) -
                              max(p["model_t_comp_us"], p["model_t_mem_us"])) < 1e-9 and
                          q["split_k"] == p["split_k"])
            if same_total:
                assert q["model_t_comp_us"] >= p["model_t_comp_us"] - 1e-9, (q["name"], p["name"])
    finally:
        b.gemm_force_plan(dtype, b.GEMM_KERNEL_AUTO, -1, 0)
