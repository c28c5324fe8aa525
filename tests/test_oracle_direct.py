"""Pins for the direct-convolution oracle (Sec. II.A definition).

The oracle's shifted-GEMM form is checked against three things it shares no
code with: a brute-force loop over every index, scipy.signal.correlate, and
torch.nn.functional.conv2d (a cross-correlation) in float64 on the CPU.
"""
import numpy as np
import pytest
import scipy.signal
import torch

from oracle.direct import brute_force_conv2d, direct_conv2d, direct_conv2d_points

CASES = [  # B, M, N, H, W, r, pad
    (1, 1, 1, 5, 5, 3, 0),
    (2, 3, 2, 7, 6, 3, 1),
    (1, 2, 3, 6, 9, 4, 0),
    (1, 2, 2, 8, 8, 5, 2),
    (2, 1, 2, 5, 5, 1, 0),
    (1, 2, 1, 4, 4, 4, 3),     # padding wider than the image
]


def _rand(shape, seed):
    return np.random.default_rng(seed).uniform(-1, 1, size=shape)


@pytest.mark.parametrize("case", CASES)
def test_direct_equals_brute_force(case):
    B, M, N, H, W, r, pad = case
    x, w = _rand((B, M, H, W), 1), _rand((N, M, r, r), 2)
    np.testing.assert_allclose(direct_conv2d(x, w, pad), brute_force_conv2d(x, w, pad),
                               rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("case", CASES)
def test_direct_equals_scipy_correlate(case):
    B, M, N, H, W, r, pad = case
    x, w = _rand((B, M, H, W), 3), _rand((N, M, r, r), 4)
    xp = np.pad(x, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    ref = np.zeros((B, N, H + 2 * pad - r + 1, W + 2 * pad - r + 1))
    for b in range(B):
        for n in range(N):
            for m in range(M):
                ref[b, n] += scipy.signal.correlate(xp[b, m], w[n, m], mode="valid", method="direct")
    np.testing.assert_allclose(direct_conv2d(x, w, pad), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", CASES + [(2, 8, 6, 23, 17, 7, 3), (1, 4, 4, 40, 40, 13, 6)])
def test_direct_equals_torch_conv2d_float64(case):
    B, M, N, H, W, r, pad = case
    x, w = _rand((B, M, H, W), 5), _rand((N, M, r, r), 6)
    ref = torch.nn.functional.conv2d(torch.from_numpy(x), torch.from_numpy(w), padding=pad).numpy()
    np.testing.assert_allclose(direct_conv2d(x, w, pad), ref, rtol=1e-12, atol=1e-12)


def test_direct_is_correlation_not_convolution():
    # a kernel with a single tap at (0, 1) shifts the image left by one column
    x = np.arange(12, dtype=float).reshape(1, 1, 3, 4)
    w = np.zeros((1, 1, 2, 2))
    w[0, 0, 0, 1] = 1.0
    y = direct_conv2d(x, w, 0)
    np.testing.assert_array_equal(y[0, 0], x[0, 0, :2, 1:4])


def test_direct_points_match_full():
    x, w = _rand((2, 3, 11, 9), 7), _rand((4, 3, 5, 5), 8)
    y = direct_conv2d(x, w, 2)
    rng = np.random.default_rng(9)
    pts = [(int(rng.integers(2)), int(rng.integers(4)), int(rng.integers(11)), int(rng.integers(9)))
           for _ in range(40)] + [(0, 0, 0, 0), (1, 3, 10, 8)]
    got = direct_conv2d_points(x, w, 2, pts)
    np.testing.assert_allclose(got, [y[p] for p in pts], rtol=1e-12, atol=1e-12)


def test_direct_rejects_bad_shapes():
    with pytest.raises(ValueError):
        direct_conv2d(np.zeros((1, 2, 4, 4)), np.zeros((1, 3, 3, 3)))
    with pytest.raises(ValueError):
        direct_conv2d(np.zeros((1, 1, 2, 2)), np.zeros((1, 1, 3, 3)))
