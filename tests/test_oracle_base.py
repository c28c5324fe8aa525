"""Pins for the Winograd bases used by the CPU nested reference.

Eq. 2.3's F(2,3) matrices must compute a 2-output, 3-tap correlation exactly
(eqs. 2.1-2.2); checked with exact rational inputs against the sums written
out, and in 2D against the brute-force correlation.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle.nested import base_f23, toom_cook_base

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def _fr(a):
    return np.array([[Fraction(v) for v in row] for row in a], dtype=object)


def test_f23_matches_printed_matrices():
    g = GOLDEN["eq_2_3_F23"]
    b = base_f23()
    assert (b.BT == _fr(g["BT"])).all()
    assert (b.G == _fr(g["G"])).all()
    assert (b.AT == _fr(g["AT"])).all()


def _rand_fracs(rng, n):
    return np.array([Fraction(int(rng.integers(-50, 50)), int(rng.integers(1, 9))) for _ in range(n)],
                    dtype=object)


@pytest.mark.parametrize("seed", range(5))
def test_f23_computes_correlation_1d(seed):
    b = base_f23()
    rng = np.random.default_rng(seed)
    x, w = _rand_fracs(rng, 4), _rand_fracs(rng, 3)
    y = b.AT.dot(b.G.dot(w) * b.BT.dot(x))
    assert y[0] == w[0] * x[0] + w[1] * x[1] + w[2] * x[2]
    assert y[1] == w[0] * x[1] + w[1] * x[2] + w[2] * x[3]


def test_f23_computes_correlation_2d():
    # eq. 2.1: y = A^T (B^T x B (.) G w G^T) A on a 4x4 tile and 3x3 kernel
    b = base_f23()
    rng = np.random.default_rng(11)
    x = _rand_fracs(rng, 16).reshape(4, 4)
    w = _rand_fracs(rng, 9).reshape(3, 3)
    y = b.AT.dot((b.BT.dot(x).dot(b.BT.T) * b.G.dot(w).dot(b.G.T))).dot(b.AT.T)
    for i in range(2):
        for j in range(2):
            assert y[i, j] == sum(w[u, v] * x[i + u, j + v] for u in range(3) for v in range(3))


BASES = [(2, 2, [0, 1]), (2, 3, [0, 1, -1]), (3, 3, [0, 1, -1, 2]),
         (4, 3, [0, 1, -1, 2, -2]), (4, 4, [0, 1, -1, 2, -2, Fraction(1, 2)])]


@pytest.mark.parametrize("m,r,pts", BASES)
def test_toom_cook_bases_compute_correlation(m, r, pts):
    b = toom_cook_base(m, r, pts)
    rng = np.random.default_rng(m * 10 + r)
    for _ in range(3):
        x, w = _rand_fracs(rng, m + r - 1), _rand_fracs(rng, r)
        y = b.AT.dot(b.G.dot(w) * b.BT.dot(x))
        for i in range(m):
            assert y[i] == sum(w[k] * x[i + k] for k in range(r))


def test_toom_cook_reproduces_f23_up_to_point_scaling():
    # the printed F(2,3) is the points {0, 1, -1, inf} construction with each
    # Winograd point rescaled; the product of the three scalings is 1 per point
    tc, pr = toom_cook_base(2, 3, [0, 1, -1]), base_f23()
    for p in range(4):
        ka = next(pr.AT[i, p] / tc.AT[i, p] for i in range(2) if tc.AT[i, p] != 0)
        kg = next(pr.G[p, j] / tc.G[p, j] for j in range(3) if tc.G[p, j] != 0)
        kb = next(pr.BT[p, j] / tc.BT[p, j] for j in range(4) if tc.BT[p, j] != 0)
        assert (pr.AT[:, p] == ka * tc.AT[:, p]).all()
        assert (pr.G[p] == kg * tc.G[p]).all()
        assert (pr.BT[p] == kb * tc.BT[p]).all()
        assert ka * kg * kb == 1
