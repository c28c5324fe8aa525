"""Closed-form multiplication complexities -- TEST INFRASTRUCTURE ONLY.

Sec. III.C defines the multiplication complexity as the number of general
multiplications per output element; additions and multiplications by
constants in the transforms are overhead and not counted.  All figures here
are per output element and per (input channel, output channel) pair, for a
2D R x R kernel on an unbounded input, which is the square of the 1D figure.

* native convolution: R^2.
* linear decomposition on F(m, r), eq. 3.2 squared: ((l/m) * ceil(R/r))^2.
  The ceiling follows the sub-kernel count ceil(R/r)^2 of Sec. II.B; with
  R/r alone eq. 3.2 would not reproduce the paper's range.
* nested Winograd on F(m, r): l^(2n) multiplications per M_n x M_n outputs,
  with n and M_n from the level recurrence; for m = r this is eq. 3.3,
  (l/m)^(2 ceil(log_r R)).
"""
from __future__ import annotations

from fractions import Fraction

from .nested import Base, nesting_levels


def _sizes_only(m: int, r: int) -> Base:
    """A base carrying only (m, r); enough for the level recurrence."""
    return Base(m, r, None, None, None)


def native_per_output(R: int) -> Fraction:
    return Fraction(R * R)


def ld_per_output(m: int, r: int, R: int) -> Fraction:
    l = m + r - 1
    c = -(-R // r)
    return (Fraction(l, m) * c) ** 2


def nested_per_output(m: int, r: int, R: int) -> Fraction:
    lv = nesting_levels(_sizes_only(m, r), R)
    if lv.n == 0:
        return Fraction(1)
    return Fraction(lv.l ** (2 * lv.n), lv.Mn ** 2)


def nested_per_output_eq33(m: int, R: int) -> Fraction:
    """Eq. 3.3 for m = r: (l/m)^(2 ceil(log_r R)), with ceil(log_r R) computed exactly."""
    r = m
    b = 0
    while r ** b < R:
        b += 1
    return Fraction(m + r - 1, m) ** (2 * b)
