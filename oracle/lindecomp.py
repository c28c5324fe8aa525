"""Linear-decomposition Winograd on the CPU -- TEST INFRASTRUCTURE ONLY.

Sec. II.B (Fig. 2): an R x R kernel is cut into ceil(R/r)^2 non-overlapping
r x r sub-kernels (zero-padded at the end).  The input tile is h x h with
h = l + (ceil(R/r) - 1) * r; it is cut into the same number of l x l
sub-input tiles taken at stride r, which therefore overlap.  Each sub-input
tile and its sub-kernel go through F(m x m, r x r); the EWMM products of all
sub-tiles and of all M input channels are summed in the Winograd domain, and
one output transform gives an m x m output tile.  The input window then
slides by m.

Used only for the multiplication-count comparison of Sec. III.C / V.A.
"""
from __future__ import annotations

from fractions import Fraction
from typing import Optional

import numpy as np

from .nested import Base, MultCounter, _to_fractions, base_f23


def ld_conv2d(x, w, pad: int = 0, base: Optional[Base] = None, exact: bool = False,
              counter: Optional[MultCounter] = None) -> np.ndarray:
    base = base or base_f23()
    m, r, l = base.m, base.r, base.l
    BT, G, AT = (base.BT, base.G, base.AT) if exact else base.as_float()
    B, M, H, W = np.shape(x)
    N, _, R, _ = np.shape(w)
    Ho, Wo = H + 2 * pad - R + 1, W + 2 * pad - R + 1
    if Ho <= 0 or Wo <= 0:
        raise ValueError("kernel larger than the padded input")
    c = -(-R // r)                       # ceil(R/r) sub-kernels per axis
    h = l + (c - 1) * r                  # input tile per axis
    th, tw = -(-Ho // m), -(-Wo // m)
    dt = object if exact else np.float64
    zero = Fraction(0) if exact else 0.0
    if exact:
        x, w = _to_fractions(x), _to_fractions(w)
    xp = np.full((B, M, (th - 1) * m + h, (tw - 1) * m + h), zero, dtype=dt)
    xp[:, :, pad:pad + H, pad:pad + W] = x if exact else np.asarray(x, np.float64)
    wp = np.full((N, M, c * r, c * r), zero, dtype=dt)
    wp[:, :, :R, :R] = w if exact else np.asarray(w, np.float64)
    # transformed sub-kernels U[n, m, cu, cv] = G w_sub G^T
    U = np.empty((N, M, c, c, l, l), dtype=dt)
    for n in range(N):
        for mm in range(M):
            for cu in range(c):
                for cv in range(c):
                    sub = wp[n, mm, cu * r:(cu + 1) * r, cv * r:(cv + 1) * r]
                    U[n, mm, cu, cv] = G.dot(sub.dot(G.T))
    y = np.full((B, N, th * m, tw * m), zero, dtype=dt)
    for b in range(B):
        for ty in range(th):
            for tx in range(tw):
                # transformed sub-input tiles of this input tile
                Vt = np.empty((M, c, c, l, l), dtype=dt)
                for mm in range(M):
                    for cu in range(c):
                        for cv in range(c):
                            r0, c0 = ty * m + cu * r, tx * m + cv * r
                            X = xp[b, mm, r0:r0 + l, c0:c0 + l]
                            Vt[mm, cu, cv] = BT.dot(X.dot(BT.T))
                for n in range(N):
                    acc = np.full((l, l), zero, dtype=dt)
                    for mm in range(M):
                        for cu in range(c):
                            for cv in range(c):
                                acc = acc + U[n, mm, cu, cv] * Vt[mm, cu, cv]
                    if counter is not None:
                        counter.count += M * c * c * l * l
                    y[b, n, ty * m:(ty + 1) * m, tx * m:(tx + 1) * m] = AT.dot(acc.dot(AT.T))
    return y[:, :, :Ho, :Wo]
