"""Pins for nested Winograd with a different base per level (oracle/mixed.py).

* a chain of one repeated base reproduces oracle/nested.py exactly (levels,
  and y bit for bit on small integers with F(2,3));
* chains of different Toom-Cook bases equal the direct oracle exactly in
  rational arithmetic, for kernel lengths that exercise the zero padding of
  the kernel to K_n;
* the instrumented multiplication count equals prod_j l_j^2 per tile, and
  the per-output figure of a single-base chain equals the closed form of
  oracle/counts.py.
"""
import itertools

import numpy as np
import pytest

from oracle.counts import nested_per_output
from oracle.direct import direct_conv2d
from oracle.mixed import mixed_levels, mults_per_output, nested_conv2d_mixed
from oracle.nested import MultCounter, base_f23, nested_conv2d, nesting_levels, toom_cook_base

F23 = base_f23()
F22 = toom_cook_base(2, 2, [0, 1])
F33 = toom_cook_base(3, 3, [0, 1, -1, 2])
F43 = toom_cook_base(4, 3, [0, 1, -1, 2, -2])
F44 = toom_cook_base(4, 4, [0, 1, -1, 2, -2, 3])


def _ints(shape, seed):
    return np.random.default_rng(seed).integers(-2, 3, size=shape).astype(np.float64)


@pytest.mark.parametrize("base", [F23, F22, F33, F44])
def test_single_base_chain_matches_the_level_recurrence(base):
    for R in range(2, 40):
        one = nesting_levels(base, R)
        if one.n > 4:
            break
        mixed = mixed_levels([base] * 6, R)
        assert (mixed.n, mixed.strides, mixed.Mn, mixed.Kn, mixed.Ln) == \
            (one.n, one.strides, one.Mn, one.Kn, one.Ln), R


@pytest.mark.parametrize("r,pad", [(3, 1), (5, 2), (7, 0), (9, 4), (13, 6)])
def test_single_base_chain_equals_nested_oracle_bit_for_bit(r, pad):
    x, w = _ints((1, 2, 17, 15), r), _ints((2, 2, r, r), 50 + r)
    y = nested_conv2d_mixed(x, w, pad, [F23] * 4)
    assert np.array_equal(y, nested_conv2d(x, w, pad))
    assert np.array_equal(y, direct_conv2d(x, w, pad))


CHAINS = [
    ("F23,F33", [F23, F33], [4, 6, 7]),          # M_2 = 6, K_2 = 7
    ("F33,F23", [F33, F23], [4, 7, 9]),          # M_2 = 6, K_2 = 9
    ("F22,F43", [F22, F43], [3, 5, 6]),          # M_2 = 8 > K_2 = 6
    ("F44,F23", [F44, F23], [5, 8, 12]),         # M_2 = 8, K_2 = 12
    ("F23,F22,F33", [F23, F22, F33], [5, 6, 13]),  # depth 2 for 5, 3 for 6 and 13
    # the GPU's mixed nest at depth 3: M_3 = 12, K_3 = 15 (strides 1, 2, 4)
    ("F23,F23,F33", [F23, F23, F33], [8, 13, 15]),
]


@pytest.mark.parametrize("name,chain,rs", CHAINS, ids=[c[0] for c in CHAINS])
def test_mixed_chains_are_exact(name, chain, rs):
    for r in rs:
        lv = mixed_levels(chain, r)
        assert lv.Kn >= r and lv.n >= 2
        pad = (r - 1) // 2
        x, w = _ints((1, 1, 2 * lv.Mn + 3, lv.Mn + 5), r), _ints((1, 1, r, r), 10 + r)
        y = nested_conv2d_mixed(x, w, pad, chain, exact=True)
        ref = direct_conv2d(x, w, pad)
        assert y.shape == ref.shape
        assert np.array_equal(np.asarray(y, dtype=np.float64), ref), (name, r)


def test_mult_count_and_closed_form():
    chain = [F23, F33, F22]
    r = 9
    lv = mixed_levels(chain, r)
    x, w = _ints((1, 2, 20, 18), 1), _ints((3, 2, r, r), 2)
    cnt = MultCounter()
    nested_conv2d_mixed(x, w, 4, chain, counter=cnt)
    th, tw = -(-20 // lv.Mn), -(-18 // lv.Mn)
    assert cnt.count == lv.P1 ** 2 * th * tw * 2 * 3
    for base, (m, rb) in [(F23, (2, 3)), (F33, (3, 3)), (F44, (4, 4))]:
        for R in range(2, 32):
            assert mults_per_output([base] * 6, R) == nested_per_output(m, rb, R)


def test_best_mixed_chain_never_loses_to_one_base():
    pool = [F23, F33, F43, F44]
    for R in range(4, 32):
        best_single = min(mults_per_output([b] * 6, R) for b in pool)
        best_mixed = best_single
        for depth in (1, 2, 3):
            for chain in itertools.product(pool, repeat=depth):
                try:
                    best_mixed = min(best_mixed, mults_per_output(list(chain), R))
                except ValueError:
                    pass                                  # chain too short for R
        assert best_mixed <= best_single


def test_short_chain_is_an_error():
    with pytest.raises(ValueError):
        mixed_levels([F23], 5)


@pytest.mark.parametrize("r", [16, 31, 39])
def test_gpu_mixed_nest_at_depth_4_equals_direct_in_fp64(r):
    """The GPU's mixed nest F(2,3), F(2,3), F(3,3), F(3,3) (strides 1, 2, 4, 12,
    M_4 = 36, K_4 = 39, 400 points per axis): exact rationals are too slow at
    this size, so fp64 against the direct oracle, whose only error is the
    rounding of B^T's thirds and sixths (a dropped term or a wrong sign or
    index gives O(1) errors)."""
    chain = [F23, F23, F33, F33]
    lv = mixed_levels(chain, r)
    assert (lv.n, lv.strides, lv.Mn, lv.Kn, lv.P1) == (4, [1, 2, 4, 12], 36, 39, 400)
    pad = (r - 1) // 2
    x, w = _ints((1, 2, 40, 45), r), _ints((2, 2, r, r), 70 + r)
    y = nested_conv2d_mixed(x, w, pad, chain)
    ref = direct_conv2d(x, w, pad)
    assert y.shape == ref.shape
    assert np.max(np.abs(y - ref)) <= 1e-9 * np.max(np.abs(ref))
