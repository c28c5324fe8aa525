"""Multiplication counts (Sec. III.C, Sec. V.A, Table I, abstract).

The instrumented counters of the CPU nested and linear-decomposition
references must equal the closed forms, and the closed-form ratios must give
the figures the paper prints.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import counts
from oracle.direct import direct_conv2d
from oracle.lindecomp import ld_conv2d
from oracle.nested import MultCounter, base_f23, nested_conv2d, nesting_levels, toom_cook_base

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))
F33 = toom_cook_base(3, 3, [0, 1, -1, 2])


@pytest.mark.parametrize("r,H", [(3, 8), (5, 12), (7, 12), (9, 16), (13, 16)])
def test_nested_instrumented_count_equals_closed_form(r, H):
    lv = nesting_levels(base_f23(), r)
    pad = (r - 1) // 2
    M, N = 2, 3
    x = np.random.default_rng(r).integers(-2, 3, (1, M, H, H)).astype(float)
    w = np.random.default_rng(r + 1).integers(-2, 3, (N, M, r, r)).astype(float)
    c = MultCounter()
    y = nested_conv2d(x, w, pad, counter=c)
    assert np.array_equal(y, direct_conv2d(x, w, pad))
    Ho = H + 2 * pad - r + 1
    assert Ho % lv.Mn == 0
    assert Fraction(c.count, Ho * Ho * M * N) == counts.nested_per_output(2, 3, r)


@pytest.mark.parametrize("R,H", [(4, 9), (5, 9), (7, 9), (9, 12)])
def test_ld_instrumented_count_equals_closed_form(R, H):
    x = np.random.default_rng(R).integers(-2, 3, (1, 1, H, H))
    w = np.random.default_rng(R + 1).integers(-2, 3, (1, 1, R, R))
    pad = (R - 1) // 2 if R % 2 else 0
    c = MultCounter()
    y = ld_conv2d(x, w, pad, base=F33, exact=True, counter=c)
    assert np.array_equal(y.astype(float), direct_conv2d(x, w, pad))
    Ho = H + 2 * pad - R + 1
    assert Ho % 3 == 0
    assert Fraction(c.count, Ho * Ho) == counts.ld_per_output(3, 3, R)


@pytest.mark.parametrize("R,H", [(3, 8), (4, 12), (9, 17)])
def test_nested_f33_instrumented_count(R, H):
    x = np.random.default_rng(R).integers(-2, 3, (1, 1, H, H))
    w = np.random.default_rng(R + 1).integers(-2, 3, (1, 1, R, R))
    c = MultCounter()
    y = nested_conv2d(x, w, 0, base=F33, exact=True, counter=c)
    assert np.array_equal(y.astype(float), direct_conv2d(x, w, 0))
    lv = nesting_levels(F33, R)
    Ho = H - R + 1
    assert Ho % lv.Mn == 0
    assert Fraction(c.count, Ho * Ho) == counts.nested_per_output(3, 3, R)


@pytest.mark.parametrize("m", [2, 3, 4])
def test_eq_3_3_matches_recurrence_when_m_equals_r(m):
    for R in range(2, 70):
        assert counts.nested_per_output(m, m, R) == counts.nested_per_output_eq33(m, R)


def test_abstract_range_f33_4_to_31():
    g = GOLDEN["abstract_range"]
    m, r = g["base"]
    ratios = {R: counts.ld_per_output(m, r, R) / counts.nested_per_output(m, r, R)
              for R in range(g["R_min"], g["R_max"] + 1)}
    lo, hi = min(ratios.values()), max(ratios.values())
    assert round(float(lo), 1) == g["low"] and round(float(hi), 1) == g["high"]
    assert ratios[4] == lo and ratios[27] == hi


def test_native_ratio_at_4x4():
    g = GOLDEN["native_ratio_low"]
    m, r = g["base"]
    v = counts.native_per_output(g["R"]) / counts.nested_per_output(m, r, g["R"])
    assert round(float(v), 2) == g["value"]


def test_table_1_conv2d_rows_within_two_percent():
    # Table I reports measured GOPS speed-ups on the FPGA; for the dense
    # Conv2D rows the multiplication ratio predicts them to within 2 %.
    # The depth-wise row has no channel contraction and is not a count pin.
    for row in GOLDEN["table_1"]["rows"]:
        if not row["conv"].startswith("Conv2D"):
            continue
        pred = counts.ld_per_output(3, 3, row["R"]) / counts.nested_per_output(3, 3, row["R"])
        assert abs(float(pred) / row["speedup"] - 1) < 0.02
        assert abs(row["gops_nested"] / row["gops_ld"] - row["speedup"]) < 0.01
