"""Writes tests/golden/fig7_counts.json: the multiplication-complexity series
of Sec. V.A (Fig. 7: 2D kernels from 3x3 to 31x31 on F(3,3), F(4,3), F(4,4)),
computed from the oracle's closed forms only (oracle/counts.py), plus the
best chain of per-level bases (oracle/mixed.py) for each kernel size.

General multiplications per output and channel pair:
  native R^2;  linear decomposition ((l/m) ceil(R/r))^2 (eq. 3.2);
  nested l^(2n) / M_n^2 (eq. 3.3 for m = r).

Run from the repository root: python tests/golden/make_fig7_counts.py
"""
import itertools
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))

from oracle.counts import ld_per_output, native_per_output, nested_per_output  # noqa: E402
from oracle.mixed import mults_per_output  # noqa: E402
from oracle.nested import base_f23, toom_cook_base  # noqa: E402

BASES = {"F(2,3)": base_f23(), "F(3,3)": toom_cook_base(3, 3, [0, 1, -1, 2]),
         "F(4,3)": toom_cook_base(4, 3, [0, 1, -1, 2, -2]),
         "F(4,4)": toom_cook_base(4, 4, [0, 1, -1, 2, -2, 3])}


def series():
    out = {"cite": "Sec. V.A (Fig. 7 simulation: kernel sizes 3x3..31x31, bases F(3,3), F(4,3), "
                   "F(4,4)); eqs. 3.2, 3.3",
           "generator": "tests/golden/make_fig7_counts.py (oracle/counts.py, oracle/mixed.py)",
           "R": list(range(3, 32)), "per_output": {}, "best_mixed_chain": []}
    for name, (m, r) in [("F(3,3)", (3, 3)), ("F(4,3)", (4, 3)), ("F(4,4)", (4, 4)),
                         ("F(2,3)", (2, 3))]:
        out["per_output"][name] = {
            "native": [float(native_per_output(R)) for R in out["R"]],
            "ld": [float(ld_per_output(m, r, R)) for R in out["R"]],
            "nested": [float(nested_per_output(m, r, R)) for R in out["R"]]}
    names = list(BASES)
    for R in out["R"]:
        best = None
        for depth in (1, 2, 3):
            for chain in itertools.product(names, repeat=depth):
                try:
                    v = mults_per_output([BASES[c] for c in chain], R)
                except ValueError:
                    continue
                if best is None or v < best[0]:
                    best = (v, chain)
        out["best_mixed_chain"].append({"R": R, "chain": list(best[1]),
                                        "per_output": float(best[0])})
    return out


if __name__ == "__main__":
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "fig7_counts.json")
    with open(path, "w") as fh:
        json.dump(series(), fh, indent=1)
    print("wrote", path)
