"""Nested Winograd with a different base at each level -- TEST INFRASTRUCTURE ONLY.

Sec. III.B nests one base F(m, r) with itself.  The level recurrence of
``nested.py`` does not depend on the levels sharing a base: level j may use
its own F(m_j, r_j) (l_j = m_j + r_j - 1) as long as each level's stride is
chosen so that the level below it is covered without gaps.  With level 1
the innermost (stride 1):

    s_0 = 1,  M_1 = m_1,  K_1 = r_1,
    s_j = min(M_j, K_j),
    M_{j+1} = M_j + s_j (m_{j+1} - 1),  K_{j+1} = K_j + s_j (r_{j+1} - 1),

and the chain stops at the first depth n with K_n >= R.  The input slice is
reordered into D[a_1..a_n] = x[sum_j s_{j-1} a_j] with a_j < l_j and
transformed by B_1^T (x) ... (x) B_n^T; tap k of the kernel (zero-padded to
K_n) goes to the multi-index with k_j < r_j and sum_j s_{j-1} k_j = k
(greedy, outermost digit first) and is transformed by G_1 (x) ... (x) G_n;
the output tensor Y[i_1..i_n], i_j < m_j, lands at sum_j s_{j-1} i_j (the
first of any duplicate positions is kept, as in ``nested.py``).  Exactness
follows from the same index identity as for one base: every output index
i + k splits as sum_j s_{j-1} (i_j + k_j).

A tile uses prod_j l_j^2 general multiplications for M_n^2 outputs.
"""
from __future__ import annotations

from dataclasses import dataclass
from fractions import Fraction
from typing import List, Optional, Sequence

import numpy as np

from .nested import Base, MultCounter, _as, _to_fractions, ewmm


@dataclass
class MixedLevels:
    bases: List[Base]      # base of level 1 .. n
    strides: List[int]     # s_0 .. s_{n-1}
    Mn: int
    Kn: int
    Ln: int

    @property
    def n(self) -> int:
        return len(self.bases)

    @property
    def P1(self) -> int:   # Winograd points per axis
        p = 1
        for b in self.bases:
            p *= b.l
        return p


def mixed_levels(chain: Sequence[Base], R: int) -> MixedLevels:
    """Levels for a length-R kernel taking chain[0] as level 1, chain[1] as
    level 2, ... until K_n >= R.  ValueError if the chain is too short."""
    if R < 1:
        raise ValueError("kernel length must be >= 1")
    if R == 1:
        return MixedLevels([], [], 1, 1, 1)
    if not chain:
        raise ValueError("empty chain")
    b0 = chain[0]
    bases, strides, M, K = [b0], [1], b0.m, b0.r
    j = 1
    while K < R:
        if j >= len(chain):
            raise ValueError(f"chain of {len(chain)} bases covers only {K} < {R} taps")
        b = chain[j]
        s = min(M, K)
        M, K = M + s * (b.m - 1), K + s * (b.r - 1)
        bases.append(b)
        strides.append(s)
        j += 1
    return MixedLevels(bases, strides, M, K, M + K - 1)


def _digits(flat: int, radices: List[int]) -> List[int]:
    """Multi-index of ``flat`` with the first radix most significant."""
    out = []
    for rad in reversed(radices):
        out.append(flat % rad)
        flat //= rad
    return out[::-1]


def _kron(mats: List[np.ndarray]) -> np.ndarray:
    out = np.array([[Fraction(1)]], dtype=object)
    for m in mats:
        out = np.kron(out, m)
    return out


def split_tap_mixed(k: int, lv: MixedLevels) -> List[int]:
    """Tap k -> (k_1..k_n), k_j < r_j, sum_j s_{j-1} k_j = k; outermost digit
    first, each as large as allowed."""
    n = lv.n
    digits = [0] * n
    rem = k
    for j in range(n - 1, 0, -1):
        d = min(rem // lv.strides[j], lv.bases[j].r - 1)
        digits[j] = d
        rem -= d * lv.strides[j]
    if not 0 <= rem < lv.bases[0].r:
        raise ValueError(f"tap {k} cannot be split")
    digits[0] = rem
    return digits


def input_matrix(lv: MixedLevels) -> np.ndarray:
    """(B_1^T (x) ... (x) B_n^T) S, S the 0/1 map of the reordered slice
    D[a] = x[sum_j s_{j-1} a_j]: column a of the Kronecker product is added
    to column sum_j s_{j-1} a_j (the product with S, one 1 per row of S)."""
    radices = [b.l for b in lv.bases]
    K = _kron([b.BT for b in lv.bases])
    out = np.zeros((lv.P1, lv.Ln), dtype=object)
    out[:] = Fraction(0)
    for col in range(lv.P1):
        a = _digits(col, radices)
        out[:, sum(s * aj for s, aj in zip(lv.strides, a))] += K[:, col]
    return out


def kernel_matrix(lv: MixedLevels) -> np.ndarray:
    radices = [b.r for b in lv.bases]
    weights = [int(np.prod(radices[j + 1:])) for j in range(lv.n)]
    S = np.zeros((int(np.prod(radices)), lv.Kn), dtype=object)
    S[:] = Fraction(0)
    for k in range(lv.Kn):
        d = split_tap_mixed(k, lv)
        S[sum(dj * wj for dj, wj in zip(d, weights)), k] = Fraction(1)
    return _kron([b.G for b in lv.bases]).dot(S)


def output_matrix(lv: MixedLevels) -> np.ndarray:
    radices = [b.m for b in lv.bases]
    AT = _kron([b.AT for b in lv.bases])
    out = np.zeros((lv.Mn, lv.P1), dtype=object)
    out[:] = Fraction(0)
    seen = set()
    for row in range(int(np.prod(radices))):
        i = _digits(row, radices)
        pos = sum(s * ij for s, ij in zip(lv.strides, i))
        if pos in seen:
            continue
        seen.add(pos)
        out[pos] = AT[row]
    if len(seen) != lv.Mn:
        raise ValueError("output positions do not cover the tile")
    return out


def nested_conv2d_mixed(x, w, pad: int, chain: Sequence[Base], exact: bool = False,
                        counter: Optional[MultCounter] = None) -> np.ndarray:
    """Stride-1 2D correlation by nested Winograd with per-level bases (the
    same chain along rows and columns).  Returns y[B][N][Ho][Wo]."""
    B, M, H, W = np.shape(x)
    N, Mw, r, r2 = np.shape(w)
    if Mw != M or r != r2:
        raise ValueError("shape mismatch")
    Ho, Wo = H + 2 * pad - r + 1, W + 2 * pad - r + 1
    if Ho <= 0 or Wo <= 0:
        raise ValueError("kernel larger than the padded input")
    if exact:
        x, w = _to_fractions(x), _to_fractions(w)
    dt = object if exact else np.float64
    lv = mixed_levels(chain, r)
    if lv.n == 0:
        raise ValueError("1x1 kernels need no transform")
    Mn, Ln, P1 = lv.Mn, lv.Ln, lv.P1
    IB, KG, OA = (_as(m, exact) for m in (input_matrix(lv), kernel_matrix(lv), output_matrix(lv)))
    th, tw = -(-Ho // Mn), -(-Wo // Mn)
    # kernel transform: pad to K_n x K_n at the end
    wp = np.zeros((N, M, lv.Kn, lv.Kn), dtype=dt)
    if exact:
        wp[:] = Fraction(0)
    wp[:, :, :r, :r] = w if exact else np.asarray(w, np.float64)
    U = np.empty((N, M, P1, P1), dtype=dt)
    for n in range(N):
        for m in range(M):
            U[n, m] = KG.dot(wp[n, m].dot(KG.T))
    # input transform: tiles of L_n x L_n at stride M_n, zero outside the image
    Hp, Wp = (th - 1) * Mn + Ln, (tw - 1) * Mn + Ln
    xp = np.zeros((B, M, max(Hp, H + pad), max(Wp, W + pad)), dtype=dt)
    if exact:
        xp[:] = Fraction(0)
    xp[:, :, pad:pad + H, pad:pad + W] = x if exact else np.asarray(x, np.float64)
    V = np.empty((B, th, tw, M, P1, P1), dtype=dt)
    for b in range(B):
        for ty in range(th):
            for tx in range(tw):
                for m in range(M):
                    X = xp[b, m, ty * Mn:ty * Mn + Ln, tx * Mn:tx * Mn + Ln]
                    V[b, ty, tx, m] = IB.dot(X.dot(IB.T))
    Yh = ewmm(U, V, counter)
    y = np.zeros((B, N, th * Mn, tw * Mn), dtype=dt)
    for b in range(B):
        for ty in range(th):
            for tx in range(tw):
                for n in range(N):
                    y[b, n, ty * Mn:(ty + 1) * Mn, tx * Mn:(tx + 1) * Mn] = \
                        OA.dot(Yh[b, ty, tx, n].dot(OA.T))
    return y[:, :, :Ho, :Wo]


def mults_per_output(chain: Sequence[Base], R: int) -> Fraction:
    """General multiplications per output and channel pair: prod l_j^2 / M_n^2."""
    lv = mixed_levels(chain, R)
    return Fraction(lv.P1 ** 2, lv.Mn ** 2)
