"""Pins for the CPU nested-Winograd reference.

In exact arithmetic nested Winograd is the direct convolution.  With small
integer inputs every intermediate of the F(2,3) path is a dyadic rational far
below 2^53, so the fp64 reference must equal the direct oracle bit for bit;
other bases are checked in exact rational arithmetic.
"""
import numpy as np
import pytest

from oracle.direct import brute_force_conv2d, direct_conv2d
from oracle.nested import (base_f23, ewmm, geometry, input_transform, kernel_transform,
                           nested_conv2d, output_transform, toom_cook_base)

INT_CASES = [  # B, M, N, H, W, r, pad  (depth n from r: 1->0, 2-3->1, 4-7->2, 8-15->3, 16-31->4)
    (2, 3, 2, 7, 9, 1, 0),
    (1, 2, 3, 9, 8, 1, 2),
    (1, 2, 2, 6, 7, 2, 0),
    (2, 2, 3, 9, 10, 3, 1),
    (1, 3, 2, 16, 16, 4, 0),      # the 4x4 / 16x16 shape of the smallest workload
    (1, 2, 2, 13, 11, 5, 2),
    (2, 1, 2, 12, 12, 7, 3),
    (1, 2, 1, 19, 21, 9, 4),
    (1, 1, 2, 30, 26, 13, 6),
    (1, 1, 1, 17, 18, 15, 0),
    (1, 1, 1, 40, 37, 31, 15),
]


def _ints(shape, seed):
    return np.random.default_rng(seed).integers(-2, 3, size=shape).astype(np.float64)


@pytest.mark.parametrize("case", INT_CASES)
def test_nested_bit_exact_on_small_integers(case):
    B, M, N, H, W, r, pad = case
    x, w = _ints((B, M, H, W), 100 + r), _ints((N, M, r, r), 200 + r)
    y = nested_conv2d(x, w, pad)
    ref = direct_conv2d(x, w, pad)
    assert y.shape == ref.shape
    assert np.array_equal(y, ref)


def test_nested_equals_brute_force_tiny():
    x, w = _ints((1, 2, 8, 7), 5), _ints((2, 2, 5, 5), 6)
    assert np.array_equal(nested_conv2d(x, w, 2), brute_force_conv2d(x, w, 2))


@pytest.mark.parametrize("case", [(1, 3, 4, 20, 23, 7, 3), (2, 4, 3, 30, 30, 13, 6)])
def test_nested_fp64_close_on_real_inputs(case):
    B, M, N, H, W, r, pad = case
    rng = np.random.default_rng(7)
    x, w = rng.standard_normal((B, M, H, W)), rng.standard_normal((N, M, r, r))
    y, ref = nested_conv2d(x, w, pad), direct_conv2d(x, w, pad)
    assert np.linalg.norm(y - ref) / np.linalg.norm(ref) < 1e-12


@pytest.mark.parametrize("m,r,pts,R", [
    (3, 3, [0, 1, -1, 2], 5), (3, 3, [0, 1, -1, 2], 10), (4, 3, [0, 1, -1, 2, -2], 7),
    (4, 4, [0, 1, -1, 2, -2, 3], 6), (2, 2, [0, 1], 4), (2, 2, [0, 1], 5)])
def test_nested_exact_other_bases(m, r, pts, R):
    base = toom_cook_base(m, r, pts)
    x = np.random.default_rng(R).integers(-3, 4, size=(1, 2, R + 5, R + 3))
    w = np.random.default_rng(R + 1).integers(-3, 4, size=(2, 2, R, R))
    y = nested_conv2d(x, w, 1, base=base, exact=True)
    assert np.array_equal(y.astype(np.float64), direct_conv2d(x, w, 1))


def test_stage_shapes_and_composition():
    x, w = _ints((2, 3, 11, 10), 1), _ints((4, 3, 7, 7), 2)
    g = geometry(x.shape, w.shape, 3)
    U = kernel_transform(w, g)
    V = input_transform(x, g)
    Yh = ewmm(U, V)
    assert g.lv.n == 2 and (g.th, g.tw) == (3, 3)
    assert U.shape == (4, 3, 16, 16) and V.shape == (2, 3, 3, 3, 16, 16) and Yh.shape == (2, 3, 3, 4, 16, 16)
    assert np.array_equal(output_transform(Yh, g), direct_conv2d(x, w, 3))
