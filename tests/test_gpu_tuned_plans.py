"""Every measured plan of the decode and prefill shapes (M <= 2048), run at its own shape,
and the plans that other row counts up to 2048 borrow from them (needs an MI355X).

The tuned plan table maps exact shapes to (configuration, split, reduction); these are
the plans a caller of those shapes gets, and a shape with M <= 2048 and no plan of its own
at the same N and K borrows the one of the nearest tuned M with as many tile rows.  Each is run through the C ABI
with the selector's own choice (no override), on seeded inputs, and compared with the
oracle: int8 element by element, bf16 by the normalised error; the whole C up to 64 rows,
sampled rows above (int8 also by Freivalds' test over the whole C).  Larger shapes of the
table are the benchmark's workloads, covered at full size by the parity tests of each B
layout.  Tests of one (dtype, K, N) run back to back and share one B.
"""
import functools
import os
import re

import numpy as np
import pytest

from oracle import oracle
from paper_2512_13282_amd import binding as b
from paper_2512_13282_amd import inputs
import gpu_helpers as g

pytestmark = pytest.mark.gpu
I8, BF = g.I8, g.BF


def _entries():
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                        "paper_2512_13282_amd", "csrc", "tuned_plans.inc")
    out = []
    for line in open(path):
        m = re.match(r"\s*\{(\d+), (\d+), (\d+), (\d+), (\d+), (\d+), (-?\d+), ([01])\},", line)
        if m:
            out.append(tuple(int(x) for x in m.groups()))
    return out


_order = lambda e: (e[0], e[3], e[2], e[-1], e[1])     # dtype, K, N, layout, M
TABLE_ENTRIES = sorted((e for e in _entries() if e[1] <= 2048), key=_order)
# (dtype, M, N, K, B layout) at each (dtype, layout, N, K) with skinny tuned plans, for row
# counts without a plan of their own
_GROUPS = {(e[0], e[2], e[3], e[7]) for e in TABLE_ENTRIES if e[1] <= 64}
BORROWED = sorted({(d, M, N, K, bt) for (d, N, K, bt) in _GROUPS for M in (3, 12, 40, 96, 192, 480, 2000)} -
                  {(e[0], e[1], e[2], e[3], e[7]) for e in TABLE_ENTRIES}, key=_order)
FULL_ROWS = 64


@pytest.fixture(autouse=True)
def _reset_plan():
    g.unforce()
    yield
    g.unforce()


@functools.lru_cache(maxsize=1)
def _b(d, K, N):
    """B (K x N) of one (dtype, K, N), and its transpose, drawn once for the tests that share it."""
    B = (inputs.int8_matrix if d == I8 else inputs.bf16_matrix)(K, N, seed=1 + K + N)
    return B, np.ascontiguousarray(B.T)


def _run_and_check(d, M, N, K, bt, seed):
    fake = 1 << 40
    plan = b.gemm_plan(d, M, N, K, K, K if bt else N, N, fake, 2 * fake, 3 * fake, trans_b=bool(bt))
    print(f"dtype={d} M={M} K={K} N={N} bt={bt} plan={plan['name']} split={plan['split_k']} "
          f"reduce={plan['reduce_in_kernel']}", flush=True)
    A = (inputs.int8_matrix if d == I8 else inputs.bf16_matrix)(M, K, seed=seed)
    B, Bt = _b(d, K, N)
    C = np.ascontiguousarray(g.gemm_gpu_bt(d, A, Bt) if bt else g.gemm_gpu(d, A, B))
    if M <= FULL_ROWS:
        (g.check_i8 if d == I8 else g.check_bf16)(A, B, C)
        return plan
    rng = np.random.default_rng(seed)
    rows = sorted({0, M // 2, M - 1} | {int(r) for r in rng.integers(0, M, size=5)})
    Ar = np.ascontiguousarray(A[rows])
    if d == I8:
        assert oracle.get().freivalds_i8_i32(A, B, C, trials=2) == 0
        g.check_i8(Ar, B, np.ascontiguousarray(C[rows]))
    else:
        assert np.all(np.isfinite(C))
        g.check_bf16(Ar, B, np.ascontiguousarray(C[rows]))
    return plan


def test_table_has_short_entries():
    assert sum(e[1] <= 64 for e in TABLE_ENTRIES) >= 40 and len(_GROUPS) >= 20 and len(TABLE_ENTRIES) >= 300


@pytest.mark.parametrize("entry", TABLE_ENTRIES,
                         ids=[f"{'i8' if e[0] == I8 else 'bf16'}-{e[1]}x{e[3]}x{e[2]}{'-bt' if e[7] else ''}"
                              for e in TABLE_ENTRIES])
def test_tuned_plan_at_its_shape(entry):
    d, M, N, K, cfg, split, reduce, bt = entry
    plan = _run_and_check(d, M, N, K, bt, seed=M)
    assert plan["config"] == cfg and plan["split_k"] == split, plan
    if reduce >= 0 and split > 1:
        assert plan["reduce_in_kernel"] == reduce, plan


@pytest.mark.parametrize("shape", BORROWED,
                         ids=[f"{'i8' if s[0] == I8 else 'bf16'}-{s[1]}x{s[3]}x{s[2]}{'-bt' if s[4] else ''}"
                              for s in BORROWED])
def test_borrowed_plan(shape):
    d, M, N, K, bt = shape
    _run_and_check(d, M, N, K, bt, seed=M + 1)
