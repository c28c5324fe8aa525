"""Pins for the depthwise oracle (Table I's depth-wise row: one kernel per
channel, no sum over channels).

* the direct depthwise definition against nested Python loops (tiny inputs);
* against the dense direct oracle with a block-diagonal weight, where
  w_dense[n][m] = w[n] if n == m else 0 -- the same operation through the
  already pinned channel-summing path;
* the nested depthwise reference bit-exact against it on small integers
  (dyadic F(2,3) intermediates), depths 0 to 4;
* its multiplication count: one general multiplication per point, tile and
  channel (the element-wise product has no channel sum).
"""
import numpy as np
import pytest

from oracle.direct import direct_conv2d, direct_depthwise_conv2d
from oracle.nested import (MultCounter, depthwise_geometries, ewmm_depthwise, input_transform,
                           kernel_transform, nested_depthwise_conv2d, output_transform)


def _ints(shape, seed):
    return np.random.default_rng(seed).integers(-2, 3, size=shape).astype(np.float64)


def _loops(x, w, pad):
    B, C, H, W = x.shape
    r = w.shape[2]
    Ho, Wo = H + 2 * pad - r + 1, W + 2 * pad - r + 1
    y = np.zeros((B, C, Ho, Wo))
    for b in range(B):
        for c in range(C):
            for i in range(Ho):
                for j in range(Wo):
                    s = 0.0
                    for u in range(r):
                        for v in range(r):
                            ii, jj = i + u - pad, j + v - pad
                            if 0 <= ii < H and 0 <= jj < W:
                                s += x[b, c, ii, jj] * w[c, 0, u, v]
                    y[b, c, i, j] = s
    return y


@pytest.mark.parametrize("B,C,H,W,r,pad", [(1, 2, 5, 6, 1, 0), (2, 3, 6, 5, 2, 0),
                                           (1, 2, 7, 7, 3, 1), (1, 3, 8, 6, 5, 2),
                                           (2, 1, 4, 4, 4, 2)])
def test_direct_depthwise_matches_loops(B, C, H, W, r, pad):
    rng = np.random.default_rng(B * 100 + C * 10 + r)
    x = rng.standard_normal((B, C, H, W))
    w = rng.standard_normal((C, 1, r, r))
    np.testing.assert_allclose(direct_depthwise_conv2d(x, w, pad), _loops(x, w, pad),
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("r,pad", [(1, 0), (3, 1), (7, 3), (4, 0)])
def test_direct_depthwise_is_dense_conv_with_diagonal_weights(r, pad):
    rng = np.random.default_rng(r)
    C = 5
    x = rng.standard_normal((2, C, 11, 9))
    w = rng.standard_normal((C, 1, r, r))
    wd = np.zeros((C, C, r, r))
    for c in range(C):
        wd[c, c] = w[c, 0]
    np.testing.assert_allclose(direct_depthwise_conv2d(x, w, pad), direct_conv2d(x, wd, pad),
                               rtol=1e-12, atol=1e-12)


DW_INT = [(2, 3, 7, 9, 1, 0), (1, 2, 9, 8, 1, 1), (2, 3, 9, 10, 3, 1), (1, 4, 16, 16, 4, 0),
          (1, 3, 13, 11, 7, 3), (1, 2, 19, 21, 9, 4), (1, 2, 17, 18, 15, 0),
          (1, 1, 40, 37, 31, 15)]


@pytest.mark.parametrize("case", DW_INT)
def test_nested_depthwise_bit_exact_on_small_integers(case):
    B, C, H, W, r, pad = case
    x, w = _ints((B, C, H, W), 300 + r), _ints((C, 1, r, r), 400 + r)
    y = nested_depthwise_conv2d(x, w, pad)
    ref = direct_depthwise_conv2d(x, w, pad)
    assert y.shape == ref.shape
    assert np.array_equal(y, ref)


def test_nested_depthwise_stages_and_count():
    B, C, H, W, r, pad = 1, 3, 12, 10, 5, 2
    x, w = _ints((B, C, H, W), 1), _ints((C, 1, r, r), 2)
    gk, gx = depthwise_geometries(x.shape, w.shape, pad)
    assert (gk.M, gk.N, gx.M, gx.N) == (1, C, C, C)
    U = kernel_transform(w, gk)
    V = input_transform(x, gx)
    cnt = MultCounter()
    Yh = ewmm_depthwise(U, V, cnt)
    P = gx.lv.P1 ** 2
    assert cnt.count == P * B * gx.th * gx.tw * C
    assert np.array_equal(output_transform(Yh, gx), direct_depthwise_conv2d(x, w, pad))


def test_depthwise_shape_errors():
    with pytest.raises(ValueError):
        direct_depthwise_conv2d(np.zeros((1, 3, 5, 5)), np.zeros((3, 2, 3, 3)))
    with pytest.raises(ValueError):
        depthwise_geometries((1, 3, 5, 5), (2, 1, 3, 3), 0)
