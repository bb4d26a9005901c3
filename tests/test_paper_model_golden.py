"""The paper's printed tile-model values reproduce under our reading of its equations.

Fixture: tests/golden/paper_tile_models.txt (single-core table and the two
array tables of Sec. 5).  Checked:

* Eq. 5 (L1 footprint: double-buffered A and B, single C) against the printed
  "L1 Core Mem." column, to the printed 0.1 KB (one row of the XDNA2 array
  table, int8-int32 128x56x80, prints 62.3 KB where Eq. 5 gives 62.75 KB: a
  known inconsistency in the paper, listed as such);
* the peak convention TOPS = 2 * MACs/cycle * cores * f against the printed
  "Peak Comp. TOPS" column.  The MACs/cycle column is itself printed to 0.1
  and two peak entries look truncated rather than rounded (6.6368 printed as
  6.63, 39.5136 as 39.52), so the bound is one printed unit (0.01 TOPS) plus
  the MACs rounding (0.05 MACs/cycle scaled to the array).
"""
import os

import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_tile_models.txt")
TY = {"int8": 1, "int16": 2, "int32": 4, "bf16": 2}
ARRAY = {"XDNA": (16, 1.0e9), "XDNA2": (32, 1.8e9)}
KNOWN_INCONSISTENT = {("T3", "int8-int32", 128, 56, 80)}


def rows():
    out = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        t, dev, io, m, k, n, macs, l1, peak = line.split()
        out.append((t, dev, io, int(m), int(k), int(n), float(macs), float(l1),
                    None if peak == "-" else float(peak)))
    return out


def eq5_l1_kb(m, k, n, ty_a, ty_b, ty_c):
    return (2 * m * k * ty_a + 2 * k * n * ty_b + m * n * ty_c) / 1024.0


@pytest.mark.parametrize("row", rows(), ids=lambda r: f"{r[0]}-{r[1]}-{r[2]}-{r[3]}x{r[4]}x{r[5]}")
def test_eq5_l1_footprint(row):
    t, dev, io, m, k, n, macs, l1, peak = row
    tin, tout = io.split("-")
    kb = eq5_l1_kb(m, k, n, TY[tin], TY[tin], TY[tout])
    assert kb <= 63.0                                   # Eq. 5's 63 KB budget
    if (t, io, m, k, n) in KNOWN_INCONSISTENT:
        assert abs(kb - 62.75) < 1e-9 and l1 == 62.3
    else:
        assert abs(kb - l1) <= 0.051, (kb, l1)


@pytest.mark.parametrize("row", [r for r in rows() if r[8] is not None],
                         ids=lambda r: f"{r[0]}-{r[1]}-{r[2]}-{r[3]}x{r[4]}x{r[5]}")
def test_peak_tops_convention(row):
    t, dev, io, m, k, n, macs, l1, peak = row
    cores, f = ARRAY[dev]
    tops = 2 * macs * cores * f / 1e12
    bound = 0.01 + 2 * 0.05 * cores * f / 1e12
    assert abs(tops - peak) <= bound, (tops, peak)
