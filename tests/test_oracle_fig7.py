"""The Fig. 7 multiplication series (Sec. V.A) from the oracle's closed forms.

tests/golden/fig7_counts.json is written by tests/golden/make_fig7_counts.py,
which calls only oracle/; this test re-derives it and checks the properties
the text states about the curves.
"""
import json
import os
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))

import make_fig7_counts  # noqa: E402

from oracle.counts import nested_per_output  # noqa: E402


@pytest.fixture(scope="module")
def stored():
    with open(os.path.join(HERE, "golden", "fig7_counts.json")) as fh:
        return json.load(fh)


def test_stored_series_is_what_the_oracle_gives(stored):
    assert make_fig7_counts.series() == stored


def test_nested_steps_at_powers_of_r():
    # Sec. V.A: the zig-zag comes from padding the kernel to a power of r
    # (m = r bases): the nested count is constant on (r^k, r^(k+1)] and jumps
    # right after each power
    for m in (3, 4):
        r = m
        for R in range(2, 32):
            k = 0
            while r ** (k + 1) < R:
                k += 1
            lo = r ** k + 1
            assert nested_per_output(m, r, R) == nested_per_output(m, r, max(lo, 2))
        for k in (1, 2):
            if r ** k + 1 <= 31:
                assert nested_per_output(m, r, r ** k + 1) > nested_per_output(m, r, r ** k)


def test_gap_to_linear_decomposition_grows_with_kernel_size(stored):
    # the F(3,3) advantage over linear decomposition at the end of the range
    # exceeds the one at the start
    po = stored["per_output"]["F(3,3)"]
    ratio = [l / n for l, n in zip(po["ld"], po["nested"])]
    assert ratio[0] == 1.0                       # R = 3: one level, same algorithm
    assert max(ratio[-8:]) > 3 * ratio[1]        # R = 24..31 vs R = 4


def test_best_chain_is_at_most_the_best_single_base(stored):
    for i, R in enumerate(stored["R"]):
        single = min(stored["per_output"][b]["nested"][i] for b in ("F(3,3)", "F(4,3)", "F(4,4)", "F(2,3)"))
        assert stored["best_mixed_chain"][i]["per_output"] <= single + 1e-12
