"""The test helpers that re-order the oracle's Winograd-domain arrays to the
library's documented point order (tests/layout.py), checked on the CPU.

The uniform-base permutation and the mixed-radix one are built in two
different ways; with every radix 4 they must agree.
"""
import numpy as np
import pytest

from tests.layout import mixed_to_lib_points, point_permutation, quads, to_lib_points


@pytest.mark.parametrize("n", [1, 2, 3])
def test_point_permutation_is_bijection(n):
    perm = point_permutation(n)
    assert len({tuple(p) for p in perm}) == 4 ** (2 * n)
    assert perm.min() == 0 and perm.max() == 4 ** n - 1


@pytest.mark.parametrize("n", [1, 2, 3])
def test_uniform_and_mixed_radix_orders_agree(n):
    P1 = 4 ** n
    a = np.arange(2 * P1 * P1, dtype=np.int64).reshape(2, P1, P1)
    assert np.array_equal(to_lib_points(a, n), mixed_to_lib_points(a, [4] * n))


def test_point_order_digits_by_hand():
    # depth 2: p = 64 q2r + 16 q2c + 4 q1r + q1c; the oracle's row index is
    # 4 q1r + q2r (level 1 most significant), its column 4 q1c + q2c
    perm = point_permutation(2)
    for q2r, q2c, q1r, q1c in [(0, 0, 0, 1), (1, 0, 0, 0), (3, 2, 1, 0), (2, 3, 3, 1)]:
        p = 64 * q2r + 16 * q2c + 4 * q1r + q1c
        assert tuple(perm[p]) == (4 * q1r + q2r, 4 * q1c + q2c)


def test_quads_puts_the_level1_column_digit_innermost():
    a = np.arange(8 * 2 * 3).reshape(8, 2, 3)
    q = quads(a)
    assert q.shape == (2, 2, 3, 4)
    for p in range(8):
        assert np.array_equal(q[p // 4, :, :, p % 4], a[p])
