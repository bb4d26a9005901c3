"""Planted mistakes in the oracle must be caught by its pins (CPU only).

Each mutant is a copy of ``oracle/oracle_gemm.c`` with one plausible bug (a
dropped term, a wrong index or stride, a sign/width error, a broken range
check...), compiled with gcc into a temporary directory.  The pins of
``oracle_pins.py`` run against it in a child process (a crash counts as
caught); at least one pin must fail for every mutant.
"""
import concurrent.futures as cf
import json
import os
import subprocess
import sys

import pytest

from oracle import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)

# (name, original text, replacement) -- the original must occur exactly once.
MUTANTS = [
    ("int_drop_last_k",
     "for (int64_t k = 0; k < j->K; ++k) {\n            const int64_t a",
     "for (int64_t k = 0; k < j->K - 1; ++k) {\n            const int64_t a"),
    ("bf16_drop_first_k",
     "for (int64_t k = 0; k < j->K; ++k) {\n            const double a",
     "for (int64_t k = 1; k < j->K; ++k) {\n            const double a"),
    ("int_ignore_lda",
     "const int64_t a = (int64_t)A[i * j->lda + k];",
     "const int64_t a = (int64_t)A[i * j->K + k];"),
    ("int_b_unsigned",
     "acc[c] += a * (int64_t)brow[c];",
     "acc[c] += a * (int64_t)(uint8_t)brow[c];"),
    ("int_a_shifted_k",
     "const int64_t a = (int64_t)A[i * j->lda + k];",
     "const int64_t a = (int64_t)A[i * j->lda + (k + 1) % j->K];"),
    ("int_int32_accumulator",
     "acc[c] += a * (int64_t)brow[c];",
     "acc[c] = (int32_t)(uint32_t)(uint64_t)(acc[c] + a * (int64_t)brow[c]);"),
    ("int_overflow_check_one_sided",
     "if (acc[c] < INT32_MIN || acc[c] > INT32_MAX) j->overflow++;",
     "if (acc[c] > INT32_MAX) j->overflow++;"),
    ("int_ignore_ldc",
     "int32_t *crow = (int32_t *)j->C + i * j->ldc;",
     "int32_t *crow = (int32_t *)j->C + i * j->N;"),
    ("int_b_transposed",
     "const int8_t *brow = B + k * j->ldb;\n            for (int64_t c = 0; c < j->N; ++c) acc[c] += a * (int64_t)brow[c];",
     "for (int64_t c = 0; c < j->N; ++c) acc[c] += a * (int64_t)((c < j->K && k < j->N) ? B[c * j->ldb + k] : 0);"),
    ("bf16_widen_shift",
     "uint32_t u = (uint32_t)bits << 16;",
     "uint32_t u = (uint32_t)bits << 15;"),
    ("bf16_float_accumulator",
     "for (int64_t c = 0; c < j->N; ++c) acc[c] += a * brow_d[c];",
     "for (int64_t c = 0; c < j->N; ++c) acc[c] = (float)(acc[c] + a * brow_d[c]);"),
    ("bf16_bf16_rounded_a",
     "const double a = oracle_bf16_to_double(A[i * j->lda + k]);",
     "const double a = oracle_bf16_to_double(A[i * j->lda + k] & 0xFFFE);"),
    ("thread_rows_off_by_one",
     "j->row1 = M * (t + 1) / nthreads;",
     "j->row1 = M * (t + 1) / nthreads - (t + 1 < nthreads && M * (t + 1) / nthreads > M * t / nthreads ? 1 : 0);"),
    ("requant_ties_away",
     "if (r > half || (r == half && q % 2 != 0)) q += 1;",
     "if (r >= half) q += 1;"),
    ("requant_truncates",
     "    if (shift > 0) {\n        const int64_t half",
     "    if (shift < 0) {\n        const int64_t half"),
    ("requant_no_floor",
     "if (v % d != 0 && v < 0) q -= 1;",
     "if (v % d != 0 && v > 0) q -= 0;"),
    ("requant_clamp_low_off_by_one",
     "hi = ((int64_t)1 << (bits - 1)) - 1, lo = -hi - 1;",
     "hi = ((int64_t)1 << (bits - 1)) - 1, lo = -hi;"),
    ("bf16_round_truncates",
     "const double r = nearbyint(ldexp(ax, -ulp_exp));",
     "const double r = trunc(ldexp(ax, -ulp_exp));"),
    ("bf16_round_nine_bits",
     "int ulp_exp = e - 8;",
     "int ulp_exp = e - 9;"),
    ("bf16_round_overflow_early",
     "if (y > 0x1.fep127)",
     "if (y > 0x1.fcp127)"),
    ("bf16_round_no_subnormal_floor",
     "if (ulp_exp < -133) ulp_exp = -133;",
     "if (ulp_exp < -149) ulp_exp = -149;"),
    ("bf16_round_nan_to_inf",
     "if (isnan(x)) return (uint16_t)(sign | 0x7FC0u);",
     "if (isnan(x)) return (uint16_t)(sign | 0x7F80u);"),
    ("freivalds_skip_last_row",
     "for (int64_t i = 0; i < M; ++i) {\n            __int128 lhs",
     "for (int64_t i = 0; i < M - 1; ++i) {\n            __int128 lhs"),
]

_CHILD = r"""
import json, sys
sys.path[:0] = [{root!r}, {here!r}]
from oracle import oracle
import oracle_pins
o = oracle.Oracle({lib!r})
failed = []
for p in oracle_pins.PINS:
    try:
        p(o)
    except AssertionError:
        failed.append(p.__name__)
print(json.dumps(failed))
"""


def _run_mutant(tmp, name, old, new):
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, f"mutant {name}: pattern not found exactly once"
    path = os.path.join(tmp, f"{name}.c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    lib = oracle.build(src=path, out=os.path.join(tmp, f"lib{name}.so"))
    r = subprocess.run([sys.executable, "-c", _CHILD.format(root=ROOT, here=HERE, lib=lib)],
                       capture_output=True, text=True, timeout=300)
    if r.returncode != 0:
        return name, ["<crashed>"]
    return name, json.loads(r.stdout.strip().splitlines()[-1])


def test_every_mutant_is_caught(tmp_path):
    with cf.ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda m: _run_mutant(str(tmp_path), *m), MUTANTS))
    survivors = [name for name, failed in results if not failed]
    assert not survivors, f"mutants not caught by any pin: {survivors}"


def test_unmutated_copy_passes(tmp_path):
    """Control: the unmodified source, built the same way, fails no pin."""
    name, failed = _run_mutant(str(tmp_path), "control", "#define ORACLE_OK 0", "#define ORACLE_OK 0")
    assert failed == [], failed
