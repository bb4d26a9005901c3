"""Plans loaded at run time (gemm_load_plans / GEMM_MI355X_PLANS), pure host: they take
precedence over the compiled table and the model for exactly their shapes, a file with
any bad line loads nothing, and the tuner's writer produces files that load."""
import os
import subprocess
import sys

import pytest

from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import tune

I8, BF = b.GEMM_DTYPE_I8_I32, b.GEMM_DTYPE_BF16_F32
AL = 1 << 40
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def plan(dtype, M, N, K, bt=False, off=0):
    return b.gemm_plan(dtype, M, N, K, K, K if bt else N, N, AL + off, 2 * AL, 3 * AL, trans_b=bt)


def triple(p):
    return p["config"], p["split_k"], p["reduce_in_kernel"]


@pytest.fixture(autouse=True)
def _clean():
    b.gemm_clear_plans()
    yield
    b.gemm_clear_plans()


def write(tmp_path, text, name="plans.txt"):
    path = tmp_path / name
    path.write_text(text)
    return str(path)


def test_loaded_plan_takes_precedence_and_clears(tmp_path):
    others = [(I8, 101, 1024, 3072, False), (BF, 100, 1024, 3072, False), (I8, 100, 1024, 3072, True)]
    before = triple(plan(I8, 100, 1024, 3072))
    others_before = [triple(plan(d, M, N, K, bt)) for (d, M, N, K, bt) in others]
    assert before != (30, 3, b.GEMM_REDUCE_SEPARATE)
    assert b.gemm_load_plans(write(tmp_path, "0 100 1024 3072 30 3 0 0\n")) == b.GEMM_OK
    assert triple(plan(I8, 100, 1024, 3072)) == (30, 3, b.GEMM_REDUCE_SEPARATE)
    # only that shape, dtype and layout
    assert [triple(plan(d, M, N, K, bt)) for (d, M, N, K, bt) in others] == others_before
    assert b.gemm_clear_plans() == b.GEMM_OK
    assert triple(plan(I8, 100, 1024, 3072)) == before


def test_loaded_plan_overrides_the_compiled_table(tmp_path):
    compiled = triple(plan(I8, 1, 14336, 4096))          # a shape of the compiled table
    assert compiled == (28, 4, b.GEMM_REDUCE_ATOMIC_FLAG)
    assert b.gemm_load_plans(write(tmp_path, "0 1 14336 4096 31 8 2 0\n")) == b.GEMM_OK
    assert triple(plan(I8, 1, 14336, 4096)) == (31, 8, b.GEMM_REDUCE_ATOMIC)
    # the column-major layout of the same shape keeps its own plan
    assert plan(I8, 1, 14336, 4096, bt=True)["config"] != 31
    b.gemm_clear_plans()
    assert triple(plan(I8, 1, 14336, 4096)) == compiled


def test_layouts_are_separate(tmp_path):
    row = triple(plan(BF, 48, 2048, 5120))
    assert b.gemm_load_plans(write(tmp_path, "1 48 2048 5120 30 4 1 1\n")) == b.GEMM_OK
    assert triple(plan(BF, 48, 2048, 5120, bt=True)) == (30, 4, b.GEMM_REDUCE_LAST_SLICE)
    assert triple(plan(BF, 48, 2048, 5120)) == row


def test_reductions_the_kernel_cannot_take_are_downgraded(tmp_path):
    # bf16 never adds atomically; the fill-free atomic reduction needs a ring or GEMV kernel
    text = "1 48 2048 5120 30 4 3 0\n0 300 2048 5120 10 2 3 0\n"
    assert b.gemm_load_plans(write(tmp_path, text)) == b.GEMM_OK
    assert triple(plan(BF, 48, 2048, 5120)) == (30, 4, b.GEMM_REDUCE_SEPARATE)
    assert triple(plan(I8, 300, 2048, 5120)) == (10, 2, b.GEMM_REDUCE_ATOMIC)


def test_comments_blank_lines_and_the_last_line_wins(tmp_path):
    text = ("# a comment\n\n   \n"
            "0 100 1024 3072 30 3 0 0   # trailing comment\n"
            "\t0 100 1024 3072 31 2 -1 0\r\n"
            "0 7 1024 3072 22 2 1 0")                      # no final newline
    assert b.gemm_load_plans(write(tmp_path, text)) == b.GEMM_OK
    assert triple(plan(I8, 100, 1024, 3072))[:2] == (31, 2)
    assert triple(plan(I8, 7, 1024, 3072)) == (22, 2, b.GEMM_REDUCE_LAST_SLICE)


def test_a_later_load_replaces_and_adds(tmp_path):
    assert b.gemm_load_plans(write(tmp_path, "0 100 1024 3072 30 3 0 0\n", "a.txt")) == b.GEMM_OK
    assert b.gemm_load_plans(write(tmp_path, "0 100 1024 3072 31 2 0 0\n0 9 1024 3072 22 2 0 0\n",
                                   "b.txt")) == b.GEMM_OK
    assert triple(plan(I8, 100, 1024, 3072))[:2] == (31, 2)
    assert triple(plan(I8, 9, 1024, 3072))[:2] == (22, 2)


BAD = ["0 100 1024 3072 30 3 0\n",            # seven fields
       "0 100 1024 3072 30 3 0 0 1\n",        # nine
       "0 100 1024 3072 thirty 3 0 0\n",
       "0 100 1024 3072 30.5 3 0 0\n",
       "2 100 1024 3072 30 3 0 0\n",          # dtype
       "0 -1 1024 3072 30 3 0 0\n",           # M
       "0 100 1024 3072 999 3 0 0\n",         # config
       "0 100 1024 3072 30 0 0 0\n",          # split
       "0 100 1024 3072 30 3 4 0\n",          # reduce
       "0 100 1024 3072 30 3 -2 0\n",
       "0 100 1024 3072 30 3 0 2\n",          # layout
       "0 100 1024 3072 30 3 0 0 x\n",        # trailing text
       "0 100 1024 99999999999999999999 30 3 0 0\n",
       "0 100 1024 3072 30 3 0 0 " + " " * 600 + "\n"]   # longer than a line may be


@pytest.mark.parametrize("bad", BAD, ids=[str(i) for i in range(len(BAD))])
def test_a_bad_line_loads_nothing(tmp_path, bad):
    before = triple(plan(I8, 100, 1024, 3072)), triple(plan(I8, 5, 1024, 3072))
    text = "0 5 1024 3072 30 3 0 0\n" + bad + "0 6 1024 3072 30 3 0 0\n"
    assert b.gemm_load_plans(write(tmp_path, text)) == b.GEMM_ERR_INVALID_VALUE
    assert (triple(plan(I8, 100, 1024, 3072)), triple(plan(I8, 5, 1024, 3072))) == before


def test_missing_file_and_null_path(tmp_path):
    assert b.gemm_load_plans(str(tmp_path / "absent.txt")) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_load_plans(None) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_load_plans(str(tmp_path)) == b.GEMM_ERR_INVALID_VALUE      # a directory


def test_a_plan_that_cannot_run_the_call_is_skipped(tmp_path):
    # a matrix-vector configuration for M > 1, and a vector-load configuration for a
    # misaligned operand: the selector's plan is used instead
    gemv = next(i for i in range(41) if b.gemm_force_plan(I8, b.GEMM_KERNEL_GEMV, i, 0) == b.GEMM_OK)
    b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, -1, 0)
    auto4 = triple(plan(I8, 4, 1024, 3072))
    assert b.gemm_load_plans(write(tmp_path, f"0 4 1024 3072 {gemv} 2 0 0\n0 100 1024 3072 30 3 0 0\n")) == b.GEMM_OK
    assert triple(plan(I8, 4, 1024, 3072)) == auto4
    assert plan(I8, 100, 1024, 3072, off=1)["kernel"] == b.GEMM_KERNEL_GENERIC
    assert plan(I8, 100, 1024, 3072)["config"] == 30


def test_forcing_still_wins_over_loaded_plans(tmp_path):
    assert b.gemm_load_plans(write(tmp_path, "0 100 1024 3072 30 3 0 0\n")) == b.GEMM_OK
    try:
        assert b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, 31, 2) == b.GEMM_OK
        assert plan(I8, 100, 1024, 3072)["config"] == 31
    finally:
        b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, -1, 0)
    assert plan(I8, 100, 1024, 3072)["config"] == 30


def _plan_in_child(env_value):
    code = ("from paper_2512_13282_amd import binding as b\n"
            "p = b.gemm_plan(0, 100, 1024, 3072, 3072, 1024, 1024, 1 << 40, 2 << 40, 3 << 40)\n"
            "print(p['config'], p['split_k'])\n")
    env = dict(os.environ, GEMM_MI355X_PLANS=env_value, PYTHONPATH=ROOT)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, cwd=ROOT, timeout=120)
    assert r.returncode == 0, r.stderr
    return r.stdout.split(), r.stderr


def test_environment_variable_loads_before_the_first_plan(tmp_path):
    out, err = _plan_in_child(write(tmp_path, "0 100 1024 3072 30 3 0 0\n"))
    assert out == ["30", "3"] and "not loaded" not in err
    out2, err2 = _plan_in_child(write(tmp_path, "0 100 1024 3072 30 3 9 0\n", "bad.txt"))
    assert out2 != ["30", "3"] and "not loaded" in err2


def test_the_tuner_writes_files_that_load(tmp_path):
    entries = [{"dtype": 0, "M": 100, "N": 1024, "K": 3072, "trans_b": 0, "config": 30, "split": 3, "reduce": 0,
                "name": "ring_64x128_w4_r5", "us": 12.5},
               {"dtype": 1, "M": 48, "N": 2048, "K": 5120, "trans_b": 1, "config": 20, "split": 4, "reduce": -1,
                "name": "ring_32x64_w2", "us": 30.0, "us_sustained": 28.0}]
    path = str(tmp_path / "tuned.txt")
    tune.write_plan_file(entries, path)
    assert b.gemm_load_plans(path) == b.GEMM_OK
    assert triple(plan(I8, 100, 1024, 3072)) == (30, 3, b.GEMM_REDUCE_SEPARATE)
    assert triple(plan(BF, 48, 2048, 5120, bt=True))[:2] == (20, 4)


def test_plan_source_is_reported(tmp_path):
    """gemm_plan_info.source says where each plan came from."""
    assert plan(I8, 1, 14336, 4096)["source"] == b.GEMM_PLAN_FROM_TABLE          # a shape of the table
    assert plan(I8, 3, 14336, 4096)["source"] == b.GEMM_PLAN_FROM_NEIGHBOUR      # borrows M = 1's or 8's
    assert plan(I8, 3, 14336 + 128, 4096)["source"] == b.GEMM_PLAN_FROM_MODEL    # no plans at this N
    assert plan(I8, 1, 14336, 4096, off=1)["source"] == b.GEMM_PLAN_FROM_MODEL   # misaligned: generic kernel
    assert b.gemm_load_plans(write(tmp_path, "0 100 1024 3072 30 3 0 0\n")) == b.GEMM_OK
    assert plan(I8, 100, 1024, 3072)["source"] == b.GEMM_PLAN_FROM_FILE
    try:
        assert b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, 31, 2) == b.GEMM_OK
        assert plan(I8, 100, 1024, 3072)["source"] == b.GEMM_PLAN_FROM_FORCED
    finally:
        b.gemm_force_plan(I8, b.GEMM_KERNEL_AUTO, -1, 0)
    assert plan(I8, 100, 1024, 3072)["source"] == b.GEMM_PLAN_FROM_FILE          # cached with its source
