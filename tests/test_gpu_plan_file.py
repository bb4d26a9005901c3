"""GEMM calls that run plans loaded at run time (gemm_load_plans), compared with the
oracle (needs an MI355X)."""
import numpy as np
import pytest

from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import inputs
import gpu_helpers as g

pytestmark = pytest.mark.gpu
I8, BF = g.I8, g.BF
AL = 1 << 40

# (dtype, M, N, K, B layout, config, split, reduce): plans the selector would not choose
LOADED = [(I8, 100, 1024, 3072, 0, 30, 3, b.GEMM_REDUCE_ATOMIC_FLAG),
          (I8, 100, 1040, 3072, 1, 28, 5, b.GEMM_REDUCE_SEPARATE),
          (BF, 48, 2048, 5120, 1, 20, 4, b.GEMM_REDUCE_LAST_SLICE),
          (BF, 200, 2056, 4096, 0, 31, 2, b.GEMM_REDUCE_SEPARATE)]


@pytest.fixture(autouse=True)
def _clean():
    g.unforce()
    b.gemm_clear_plans()
    yield
    b.gemm_clear_plans()


def test_loaded_plans_run_and_match_the_oracle(tmp_path):
    path = tmp_path / "plans.txt"
    path.write_text("".join(f"{d} {M} {N} {K} {cfg} {s} {r} {bt}\n" for (d, M, N, K, bt, cfg, s, r) in LOADED))
    assert b.gemm_load_plans(str(path)) == b.GEMM_OK
    for (d, M, N, K, bt, cfg, s, r) in LOADED:
        p = b.gemm_plan(d, M, N, K, K, K if bt else N, N, AL, 2 * AL, 3 * AL, trans_b=bool(bt))
        assert (p["config"], p["split_k"], p["reduce_in_kernel"]) == (cfg, s, r), p
        print(f"loaded plan dtype={d} M={M} K={K} N={N} bt={bt} {p['name']} x{s} r{r}", flush=True)
        A, B = inputs.make_inputs("int8" if d == I8 else "bf16", M, N, K, seed=M + K)
        C = g.gemm_gpu_bt(d, A, np.ascontiguousarray(B.T)) if bt else g.gemm_gpu(d, A, B)
        (g.check_i8 if d == I8 else g.check_bf16)(A, B, np.ascontiguousarray(C))
