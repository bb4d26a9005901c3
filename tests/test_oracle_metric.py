"""Pins of ``oracle.normalized_error``, the bf16 parity metric (CPU only).

The metric is max|C - C_ref| / (K * max|A| * max|B|): the absolute error of
the fp32 result against the exact fp64 sum, scaled by the largest magnitude a
single product can have times the number of products.  Every bf16 parity
verdict of the suite goes through it, so it is pinned here against values
worked out by hand, and a set of plausible mistakes in it must each fail at
least one pin.
"""
from __future__ import annotations

import inspect
import math
import textwrap

import numpy as np
import pytest

from oracle import oracle


def pin_hand_worked_value(ne):
    # diffs 0, +0.5, -1.0, 0 -> max |diff| = 1.0 ; denominator 4 * 2 * 0.5 = 4
    C = np.array([[1.0, 3.0], [1.0, 4.0]], dtype=np.float32)
    R = np.array([[1.0, 2.5], [2.0, 4.0]], dtype=np.float64)
    assert ne(C, R, 4, 2.0, 0.5) == 0.25


def pin_negative_difference_dominates(ne):
    # the largest error is negative (C below the exact value): |-4| / (3 * 1 * 1)
    C = np.array([[0.0, -3.0, 2.0]], dtype=np.float32)
    R = np.array([[0.0, 1.0, 1.0]], dtype=np.float64)
    assert ne(C, R, 3, 1.0, 1.0) == pytest.approx(4.0 / 3.0, rel=0, abs=1e-15)


def pin_max_not_mean(ne):
    # one error among many zeros: the max is 2 / (5 * 1 * 1), the mean would be 2/100 of that
    C = np.zeros((10, 10), dtype=np.float32)
    C[7, 3] = 2.0
    R = np.zeros((10, 10), dtype=np.float64)
    assert ne(C, R, 5, 1.0, 1.0) == pytest.approx(0.4, rel=0, abs=1e-15)


def pin_denominator_uses_each_factor_once(ne):
    # K = 3, max|A| = 2, max|B| = 5 -> denominator 30 (K^2 would give 90, a missing factor 6 or 15)
    C = np.array([[6.0]], dtype=np.float32)
    R = np.array([[0.0]], dtype=np.float64)
    assert ne(C, R, 3, 2.0, 5.0) == pytest.approx(0.2, rel=0, abs=1e-15)


def pin_difference_in_float64(ne):
    # C = 1 exactly (fp32), C_ref = 1 + 2^-30: the difference 2^-30 is exact in fp64 but
    # vanishes if C_ref is rounded to fp32 first
    C = np.array([[1.0]], dtype=np.float32)
    R = np.array([[1.0 + 2.0 ** -30]], dtype=np.float64)
    assert ne(C, R, 1, 1.0, 1.0) == 2.0 ** -30


def pin_zero_denominator(ne):
    # K = 0 (or an all-zero operand): the exact result is 0; C == 0 passes, anything else fails
    Z = np.zeros((2, 3), dtype=np.float32)
    R = np.zeros((2, 3), dtype=np.float64)
    assert ne(Z, R, 0, 1.0, 1.0) == 0.0
    assert ne(Z, R, 5, 0.0, 1.0) == 0.0
    C = Z.copy()
    C[1, 2] = 1e-30
    assert ne(C, R, 0, 1.0, 1.0) == math.inf
    assert ne(-C, R, 4, 1.0, 0.0) == math.inf


def pin_signed_zero_is_zero(ne):
    # -0 and +0 are the same number: no error
    C = np.array([[-0.0, 0.0]], dtype=np.float32)
    R = np.array([[0.0, -0.0]], dtype=np.float64)
    assert ne(C, R, 2, 1.0, 1.0) == 0.0


def pin_nan_fails_the_check(ne):
    # a NaN anywhere in C must never pass the 1e-5 bar
    C = np.array([[1.0, np.nan]], dtype=np.float32)
    R = np.array([[1.0, 2.0]], dtype=np.float64)
    assert not (ne(C, R, 2, 1.0, 1.0) <= 1e-5)
    assert not (ne(C, np.zeros((1, 2)), 0, 1.0, 1.0) <= 1e-5)


def pin_empty_is_zero(ne):
    assert ne(np.zeros((0, 4), dtype=np.float32), np.zeros((0, 4)), 7, 1.0, 1.0) == 0.0


PINS = [pin_hand_worked_value, pin_negative_difference_dominates, pin_max_not_mean,
        pin_denominator_uses_each_factor_once, pin_difference_in_float64, pin_zero_denominator,
        pin_signed_zero_is_zero, pin_nan_fails_the_check, pin_empty_is_zero]

# (name, original text, replacement): each original occurs exactly once in the function.
MUTANTS = [
    ("no_abs", "np.max(np.abs(C.astype(np.float64) - C_ref))", "np.max(C.astype(np.float64) - C_ref)"),
    ("mean_not_max", "np.max(np.abs(", "np.mean(np.abs("),
    ("nan_ignored", "np.max(np.abs(", "np.nanmax(np.abs("),
    ("k_squared", "float(K) * float(amax_a)", "float(K) ** 2 * float(amax_a)"),
    ("missing_amax_b", " * float(amax_b)", ""),
    ("zero_denominator_passes", 'return 0.0 if diff == 0.0 else float("inf")', "return 0.0"),
    ("diff_in_float32", "C.astype(np.float64) - C_ref", "C - C_ref.astype(np.float32)"),
    ("relative_not_normalized", "return diff / denom", "return diff / max(float(np.max(np.abs(C_ref))), 1e-300)"),
]


def _mutated(old: str, new: str):
    src = textwrap.dedent(inspect.getsource(oracle.normalized_error))
    assert src.count(old) == 1, f"mutant pattern not found exactly once: {old!r}"
    ns = {"np": np}
    exec(src.replace(old, new), ns)
    return ns["normalized_error"]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_metric_pin(pin):
    pin(oracle.normalized_error)


def test_unmutated_copy_passes():
    """Control: the function rebuilt from its own source passes every pin."""
    ne = _mutated("return diff / denom", "return diff / denom")
    for pin in PINS:
        pin(ne)


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_metric_mutant_is_caught(name, old, new):
    ne = _mutated(old, new)
    failed = []
    for pin in PINS:
        try:
            pin(ne)
        except Exception:   # a wrong value or a crash: the pin caught it
            failed.append(pin.__name__)
    assert failed, f"mutant {name} of normalized_error passes every pin"
