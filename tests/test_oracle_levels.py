"""Pins for the level recurrence, the reordering and the kernel split.

Paper values: the 1D example of Fig. 3 (Sec. III.B), the multi-level rule of
Sec. III.B, and eq. 4.1 (Sec. IV.C).
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle.nested import (base_f23, nested_input_matrix, nested_kernel_matrix,
                           nested_output_matrix, nesting_levels, split_tap, toom_cook_base)

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))
F22 = toom_cook_base(2, 2, [0, 1])


def _sizes(m, r):
    return toom_cook_base(m, r, list(range(m + r - 1))[:m + r - 2]) if (m, r) != (2, 3) else base_f23()


def test_fig3_example_geometry():
    g = GOLDEN["fig3_1d_example"]
    lv = nesting_levels(F22, g["R"])
    assert lv.n == 2
    assert lv.Ln == g["slice_length_L"]                 # L = l + r (l - 1)
    assert lv.Mn == g["slice_stride"] == g["outputs_per_slice"]
    assert lv.strides[1] == g["sub_slice_stride"]       # sub-slices at stride r
    assert lv.l ** 1 == g["reordered_matrix_side"]


def test_fig3_reordering_matches_text():
    # input reordered matrix: length-l sub-slices at stride r arranged column by column;
    # kernel reordered matrix: the length-R kernel reshaped so that horizontal
    # neighbours are r taps apart
    lv = nesting_levels(F22, 4)
    l, r = 3, 2
    x = np.array([Fraction(v) for v in [3, -1, 4, 1, -5, 9, 2]], dtype=object)
    # undo the Kronecker transform to recover the reorder alone
    from oracle.nested import _kron_all, _frac_inverse
    KB = _kron_all(F22.BT, 2)
    D = _frac_inverse(KB).dot(nested_input_matrix(F22, lv).dot(x))
    X = D.reshape(l, l)                                   # [a_1][a_2]
    for i in range(l):
        for j in range(l):
            assert X[i, j] == x[i + r * j]
    KG = _kron_all(F22.G, 2)
    w = np.array([Fraction(v) for v in [2, 7, 1, 8]], dtype=object)
    Wr = (np.linalg.pinv(KG.astype(float)) @ nested_kernel_matrix(F22, lv).dot(w).astype(float)).reshape(r, r)
    for i in range(r):
        for j in range(r):
            assert abs(Wr[i, j] - float(w[i + r * j])) < 1e-12


def test_fig3_example_computes_four_outputs():
    lv = nesting_levels(F22, 4)
    rng = np.random.default_rng(3)
    x = np.array([Fraction(int(v)) for v in rng.integers(-9, 9, 7)], dtype=object)
    w = np.array([Fraction(int(v)) for v in rng.integers(-9, 9, 4)], dtype=object)
    y = nested_output_matrix(F22, lv).dot(nested_kernel_matrix(F22, lv).dot(w)
                                          * nested_input_matrix(F22, lv).dot(x))
    assert len(y) == 4
    for i in range(4):
        assert y[i] == sum(w[k] * x[i + k] for k in range(4))


@pytest.mark.parametrize("r,n", GOLDEN["multi_level_rule"]["cases"])
def test_multi_level_rule_m_equals_r(r, n):
    # an n-dim transform covers kernels up to r^n, with l^n multiplications and m^n outputs
    base = toom_cook_base(r, r, list(range(2 * r - 2)))
    lv = nesting_levels(base, r ** n)
    assert lv.n == n and lv.Kn == r ** n and lv.Mn == r ** n
    assert lv.strides == [r ** j for j in range(n)]
    assert lv.l ** lv.n == (2 * r - 1) ** n
    assert nesting_levels(base, r ** n + 1).n == n + 1
    if n == 2:
        assert lv.Ln == (2 * r - 1) + r * (2 * r - 2)      # L = l + r (l - 1)


def test_eq_4_1_five_taps_one_nesting():
    g = GOLDEN["eq_4_1"]
    lv = nesting_levels(base_f23(), g["R"])
    assert lv.n == 2 and lv.Mn == g["M"] == g["m"] ** 2
    # under F(2,2) two levels cover only 4 taps, so 5 taps need a third level
    assert nesting_levels(F22, 5).n == 3


F23_TABLE = {  # n: (strides, M_n, K_n, L_n) derived from the recurrence for F(2,3)
    1: ([1], 2, 3, 4), 2: ([1, 2], 4, 7, 10), 3: ([1, 2, 4], 8, 15, 22), 4: ([1, 2, 4, 8], 16, 31, 46)}


@pytest.mark.parametrize("R,n", [(1, 0), (2, 1), (3, 1), (4, 2), (7, 2), (8, 3), (13, 3), (15, 3),
                                 (16, 4), (31, 4), (32, 5)])
def test_f23_depths(R, n):
    lv = nesting_levels(base_f23(), R)
    assert lv.n == n
    if n in F23_TABLE:
        s, M, K, L = F23_TABLE[n]
        assert (lv.strides, lv.Mn, lv.Kn, lv.Ln) == (s, M, K, L)


@pytest.mark.parametrize("m,r", [(2, 2), (2, 3), (3, 3), (4, 3), (4, 4), (3, 2), (2, 4)])
@pytest.mark.parametrize("n", [1, 2, 3, 4])
def test_split_tap_is_a_valid_injection(m, r, n):
    base = toom_cook_base(m, r, list(range(m + r - 2)))
    lv = None
    R = r
    while True:
        lv = nesting_levels(base, R)
        if lv.n >= n:
            break
        R = lv.Kn + 1
    seen = set()
    for k in range(lv.Kn):
        d = split_tap(k, lv.strides, r)
        assert all(0 <= dj < r for dj in d)
        assert sum(s * dj for s, dj in zip(lv.strides, d)) == k
        seen.add(tuple(d))
    assert len(seen) == lv.Kn
    # outputs cover 0..M_n-1 and taps cover 0..K_n-1 without gaps
    assert lv.Mn == 1 + sum(s * (m - 1) for s in lv.strides)
    assert lv.Kn == 1 + sum(s * (r - 1) for s in lv.strides)
