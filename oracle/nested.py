"""CPU nested-Winograd reference -- TEST INFRASTRUCTURE ONLY.

A plain, slow implementation of the nested Winograd algorithm of Sec. III.B,
in fp64 (numpy) or in exact rational arithmetic (``fractions.Fraction``
object arrays).  It is used to check the GPU library's intermediate stages
and to count multiplications; the end-to-end oracle is ``direct.py``.

Steps, in the paper's order:

1. Base F(m, r) (eqs. 2.1-2.3): y = A^T [ (G w) (.) (B^T x) ], l = m + r - 1.
   F(2,3) uses the matrices printed in eq. 2.3.
2. Nesting levels (Sec. III.B, multi-level paragraph; Alg. 1 read as a chain
   of n identical bases): a length-R kernel is handled by an n-dimensional
   Winograd transform.  Level j (1-based) works at stride s_{j-1}:
       s_0 = 1,  M_1 = m,  K_1 = r,
       s_j = min(M_j, K_j),  M_{j+1} = M_j + s_j (m-1),  K_{j+1} = K_j + s_j (r-1),
   and n is the smallest depth with K_n >= R.  L_n = M_n + K_n - 1 is the
   input slice length.  For m = r this gives s_j = r^j, M_n = K_n = r^n and
   L_2 = l + r (l-1), the slice length and stride m^2 of the 1D example.
3. Nested input transformation: the slice x[0..L_n) is reordered into the
   n-dim tensor D[a_1..a_n] = x[sum_j s_{j-1} a_j], a_j in [0, l), and
   transformed by B^T along every axis.
4. Nested kernel transformation: w is zero-padded at its end to K_n taps;
   each tap k is placed at one multi-index (k_1..k_n) in [0, r)^n with
   sum_j s_{j-1} k_j = k (greedy: k_n first, each digit as large as allowed);
   all other entries are zero; then G along every axis.
5. EWMM of the two transformed tensors, accumulated over the M input channels
   (Sec. II.B notes that the M channels are summed in the Winograd domain).
6. Nested output transformation: A^T along every axis gives the output
   reordered tensor Y[i_1..i_n], i_j in [0, m), flattened to
   y[sum_j s_{j-1} i_j]; where two multi-indices land on the same output
   (only when m > r) the values are equal and the first is kept.

In 2D (Fig. 4 text) the 1D nested transforms are applied to all rows, then
all columns, of each input tile, kernel and output tile.  A 2D input tile is
L_n x L_n, taken at stride M_n, and yields an M_n x M_n output tile.

The n-dim transform along all axes of an n-dim tensor is the Kronecker
product of the n base matrices acting on the flattened tensor; this module
builds each 1D nested transform as one explicit matrix (reorder, then
Kronecker product) and applies it to rows and columns with plain matrix
products.  Flattening order: a_1 is the most significant axis.

r = 1 needs no transform (n = 0): Winograd with no tile overlap reduces to
the native convolution (Sec. II.A, last paragraph).
"""
from __future__ import annotations

from dataclasses import dataclass
from fractions import Fraction
from typing import List, Optional

import numpy as np


# ---------------------------------------------------------------------------
# 1. Winograd bases
# ---------------------------------------------------------------------------

@dataclass
class Base:
    """Winograd base F(m, r): y = AT [(G w) (.) (BT x)]; matrices as Fraction arrays."""
    m: int
    r: int
    BT: np.ndarray   # l x l
    G: np.ndarray    # l x r
    AT: np.ndarray   # m x l

    @property
    def l(self) -> int:
        return self.m + self.r - 1

    def as_float(self):
        return (self.BT.astype(np.float64), self.G.astype(np.float64),
                self.AT.astype(np.float64))


def _frac_array(rows) -> np.ndarray:
    return np.array([[Fraction(v) for v in row] for row in rows], dtype=object)


def base_f23() -> Base:
    """F(2,3) with the matrices of eq. 2.3."""
    h = Fraction(1, 2)
    BT = _frac_array([[1, 0, -1, 0], [0, 1, 1, 0], [0, -1, 1, 0], [0, 1, 0, -1]])
    G = _frac_array([[1, 0, 0], [h, h, h], [h, -h, h], [0, 0, 1]])
    AT = _frac_array([[1, 1, 1, 0], [0, 1, -1, -1]])
    return Base(2, 3, BT, G, AT)


def _frac_inverse(A: np.ndarray) -> np.ndarray:
    """Exact inverse of a square Fraction matrix by Gauss-Jordan elimination."""
    n = A.shape[0]
    aug = np.empty((n, 2 * n), dtype=object)
    aug[:, :n] = A
    for i in range(n):
        for j in range(n):
            aug[i, n + j] = Fraction(int(i == j))
    for col in range(n):
        piv = next(rw for rw in range(col, n) if aug[rw, col] != 0)
        if piv != col:
            aug[[col, piv]] = aug[[piv, col]]
        aug[col] = aug[col] / aug[col, col]
        for rw in range(n):
            if rw != col and aug[rw, col] != 0:
                aug[rw] = aug[rw] - aug[rw, col] * aug[col]
    return aug[:, n:]


def toom_cook_base(m: int, r: int, points) -> Base:
    """F(m, r) from l-1 finite interpolation points plus the point at infinity.

    The paper names bases F(3,3), F(4,3), F(4,4) (Sec. V.A) but prints only
    F(2,3)'s matrices.  Construction (polynomial multiplication, transposed):
    the linear convolution s = w * d of a length-r w and a length-m d is
    V^{-1} [(G w) (.) (E d)] where G, E, V evaluate polynomials of degree
    r-1, m-1, l-1 at the points (the infinity row takes the leading
    coefficient).  Correlation is the transpose of that map for fixed w, so
    y = E^T [(G w) (.) (V^{-T} x)], i.e. AT = E^T and BT = V^{-T}.
    """
    l = m + r - 1
    pts = [Fraction(p) for p in points]
    if len(pts) != l - 1 or len(set(pts)) != l - 1:
        raise ValueError("need l-1 distinct finite points")

    def vander(cols):
        rows = [[p ** k for k in range(cols)] for p in pts]
        rows.append([Fraction(0)] * (cols - 1) + [Fraction(1)])
        return _frac_array(rows)

    G, E, V = vander(r), vander(m), vander(l)
    BT = _frac_inverse(V).T.copy()
    return Base(m, r, BT, G, E.T.copy())


# ---------------------------------------------------------------------------
# 2. Nesting levels
# ---------------------------------------------------------------------------

@dataclass
class Levels:
    n: int                 # nesting depth (0: no transform)
    strides: List[int]     # s_0 .. s_{n-1}: stride of level 1 .. n
    Mn: int                # outputs per axis per tile
    Kn: int                # kernel taps per axis after padding
    Ln: int                # input slice length per axis
    l: int                 # base input length

    @property
    def P1(self) -> int:   # Winograd points per axis
        return self.l ** self.n


def nesting_levels(base: Base, R: int) -> Levels:
    """Level recurrence for a length-R kernel on base F(m, r) (see module doc)."""
    if R < 1:
        raise ValueError("kernel length must be >= 1")
    m, r, l = base.m, base.r, base.l
    if R == 1:
        return Levels(0, [], 1, 1, 1, l)
    strides, M, K = [1], m, r
    while K < R:
        s = min(M, K)
        M, K = M + s * (m - 1), K + s * (r - 1)
        strides.append(s)
    return Levels(len(strides), strides, M, K, M + K - 1, l)


def split_tap(k: int, strides: List[int], r: int) -> List[int]:
    """Place kernel tap k at a multi-index (k_1..k_n), k_j < r, sum s_{j-1} k_j = k.

    Greedy from the outermost level: k_j = min(rem // s_{j-1}, r - 1).
    """
    n = len(strides)
    digits = [0] * n
    rem = k
    for j in range(n - 1, 0, -1):
        d = min(rem // strides[j], r - 1)
        digits[j] = d
        rem -= d * strides[j]
    if not 0 <= rem < r:
        raise ValueError(f"tap {k} cannot be split over strides {strides}")
    digits[0] = rem
    return digits


def _multi_indices(radix: int, n: int):
    """All multi-indices in [0, radix)^n, a_1 most significant."""
    if n == 0:
        return [()]
    return [tuple(int(c) for c in np.unravel_index(i, (radix,) * n))
            for i in range(radix ** n)]


def _kron_all(mat: np.ndarray, n: int) -> np.ndarray:
    out = np.array([[Fraction(1)]], dtype=object)
    for _ in range(n):
        out = np.kron(out, mat)
    return out


# ---------------------------------------------------------------------------
# 3.-6. The 1D nested transforms as explicit matrices
# ---------------------------------------------------------------------------

_CACHE = {}


def _cached(kind: str, base: Base, lv: Levels, build):
    key = (kind, base.m, base.r, tuple(base.BT.flat), tuple(base.G.flat), tuple(base.AT.flat),
           lv.n, tuple(lv.strides))
    if key not in _CACHE:
        _CACHE[key] = build()
    return _CACHE[key]


def nested_input_matrix(base: Base, lv: Levels) -> np.ndarray:
    """(l^n x L_n): reorder x[0..L_n) into D[a], then B^T on every axis."""
    return _cached("in", base, lv, lambda: _nested_input_matrix(base, lv))


def nested_kernel_matrix(base: Base, lv: Levels) -> np.ndarray:
    """(l^n x K_n): place each tap at its split multi-index, then G on every axis."""
    return _cached("ker", base, lv, lambda: _nested_kernel_matrix(base, lv))


def nested_output_matrix(base: Base, lv: Levels) -> np.ndarray:
    """(M_n x l^n): A^T on every axis, then flatten Y[i] to y[sum s_{j-1} i_j]."""
    return _cached("out", base, lv, lambda: _nested_output_matrix(base, lv))


def _nested_input_matrix(base: Base, lv: Levels) -> np.ndarray:
    S = np.zeros((lv.l ** lv.n, lv.Ln), dtype=object)
    S[:] = Fraction(0)
    for row, a in enumerate(_multi_indices(lv.l, lv.n)):
        S[row, sum(s * aj for s, aj in zip(lv.strides, a))] = Fraction(1)
    return _kron_all(base.BT, lv.n).dot(S)


def _nested_kernel_matrix(base: Base, lv: Levels) -> np.ndarray:
    S = np.zeros((base.r ** lv.n, lv.Kn), dtype=object)
    S[:] = Fraction(0)
    radix = [base.r ** (lv.n - 1 - j) for j in range(lv.n)]   # a_1 most significant
    for k in range(lv.Kn):
        digits = split_tap(k, lv.strides, base.r)
        S[sum(d * rad for d, rad in zip(digits, radix)), k] = Fraction(1)
    return _kron_all(base.G, lv.n).dot(S)


def _nested_output_matrix(base: Base, lv: Levels) -> np.ndarray:
    AT = _kron_all(base.AT, lv.n)                    # m^n x l^n
    out = np.zeros((lv.Mn, lv.l ** lv.n), dtype=object)
    out[:] = Fraction(0)
    seen = set()
    for row, i in enumerate(_multi_indices(base.m, lv.n)):
        pos = sum(s * ij for s, ij in zip(lv.strides, i))
        if pos in seen:
            continue                                  # duplicate output (m > r)
        seen.add(pos)
        out[pos] = AT[row]
    if len(seen) != lv.Mn:
        raise ValueError("output positions do not cover the tile")
    return out


def _as(mat: np.ndarray, exact: bool) -> np.ndarray:
    return mat if exact else mat.astype(np.float64)


# ---------------------------------------------------------------------------
# Stages in 2D
# ---------------------------------------------------------------------------

@dataclass
class Geometry:
    base: Base
    lv: Levels
    B: int
    M: int
    N: int
    H: int
    W: int
    r: int
    pad: int
    Ho: int
    Wo: int
    th: int   # tile rows per image
    tw: int   # tile columns per image


def geometry(x_shape, w_shape, pad: int, base: Optional[Base] = None) -> Geometry:
    base = base or base_f23()
    B, M, H, W = x_shape
    N, Mw, r, r2 = w_shape
    if Mw != M or r != r2:
        raise ValueError("shape mismatch")
    Ho, Wo = H + 2 * pad - r + 1, W + 2 * pad - r + 1
    if Ho <= 0 or Wo <= 0:
        raise ValueError("kernel larger than the padded input")
    lv = nesting_levels(base, r)
    th, tw = -(-Ho // lv.Mn), -(-Wo // lv.Mn)
    return Geometry(base, lv, B, M, N, H, W, r, pad, Ho, Wo, th, tw)


def kernel_transform(w, g: Geometry, exact: bool = False) -> np.ndarray:
    """U[n][m] = KG . Wpad . KG^T (rows then columns); shape (N, M, P1, P1)."""
    KG = _as(nested_kernel_matrix(g.base, g.lv), exact)
    dt = object if exact else np.float64
    wp = np.zeros((g.N, g.M, g.lv.Kn, g.lv.Kn), dtype=dt)
    if exact:
        wp[:] = Fraction(0)
    wp[:, :, :g.r, :g.r] = w if exact else np.asarray(w, dtype=np.float64)
    U = np.empty((g.N, g.M, g.lv.P1, g.lv.P1), dtype=dt)
    for n in range(g.N):
        for m in range(g.M):
            U[n, m] = KG.dot(wp[n, m].dot(KG.T))
    return U


def padded_input(x, g: Geometry, exact: bool = False) -> np.ndarray:
    """x zero-padded by pad on the top/left and enough on the bottom/right for whole tiles."""
    dt = object if exact else np.float64
    Hp = (g.th - 1) * g.lv.Mn + g.lv.Ln
    Wp = (g.tw - 1) * g.lv.Mn + g.lv.Ln
    xp = np.zeros((g.B, g.M, max(Hp, g.H + g.pad), max(Wp, g.W + g.pad)), dtype=dt)
    if exact:
        xp[:] = Fraction(0)
    xp[:, :, g.pad:g.pad + g.H, g.pad:g.pad + g.W] = x if exact else np.asarray(x, np.float64)
    return xp


def input_transform(x, g: Geometry, exact: bool = False) -> np.ndarray:
    """V[b,ty,tx,m] = IB . X_tile . IB^T for each L_n x L_n tile; shape (B, th, tw, M, P1, P1).

    Tile (ty, tx) starts at row ty*M_n - pad, column tx*M_n - pad of x.
    """
    IB = _as(nested_input_matrix(g.base, g.lv), exact)
    xp = padded_input(x, g, exact)
    dt = object if exact else np.float64
    Mn, Ln, P1 = g.lv.Mn, g.lv.Ln, g.lv.P1
    V = np.empty((g.B, g.th, g.tw, g.M, P1, P1), dtype=dt)
    for b in range(g.B):
        for ty in range(g.th):
            for tx in range(g.tw):
                for m in range(g.M):
                    X = xp[b, m, ty * Mn:ty * Mn + Ln, tx * Mn:tx * Mn + Ln]
                    V[b, ty, tx, m] = IB.dot(X.dot(IB.T))
    return V


class MultCounter:
    """Counts the general multiplications of the EWMM (Sec. III.C counts only those)."""

    def __init__(self):
        self.count = 0


def ewmm(U, V, counter: Optional[MultCounter] = None) -> np.ndarray:
    """Yhat[b,ty,tx,n] = sum_m U[n,m] (.) V[b,ty,tx,m]; shape (B, th, tw, N, P1, P1)."""
    B, th, tw, M, P1, _ = V.shape
    N = U.shape[0]
    Yh = np.empty((B, th, tw, N, P1, P1), dtype=V.dtype)
    for b in range(B):
        for ty in range(th):
            for tx in range(tw):
                for n in range(N):
                    acc = U[n, 0] * V[b, ty, tx, 0]
                    for m in range(1, M):
                        acc = acc + U[n, m] * V[b, ty, tx, m]
                    Yh[b, ty, tx, n] = acc
                    if counter is not None:
                        counter.count += M * P1 * P1
    return Yh


def ewmm_depthwise(U, V, counter: Optional[MultCounter] = None) -> np.ndarray:
    """Depthwise EWMM: Yhat[b,ty,tx,c] = U[c,0] (.) V[b,ty,tx,c], no channel sum.

    U has shape (C, 1, P1, P1) (the kernel transform of w [C][1][r][r]).
    """
    B, th, tw, C, P1, _ = V.shape
    if U.shape[:2] != (C, 1):
        raise ValueError("depthwise U must be (C, 1, P1, P1)")
    Yh = np.empty_like(V)
    for b in range(B):
        for ty in range(th):
            for tx in range(tw):
                for c in range(C):
                    Yh[b, ty, tx, c] = U[c, 0] * V[b, ty, tx, c]
                    if counter is not None:
                        counter.count += P1 * P1
    return Yh


def output_transform(Yh, g: Geometry, exact: bool = False) -> np.ndarray:
    """y tile = OA . Yhat . OA^T (M_n x M_n), placed at (ty*M_n, tx*M_n), cropped to Ho x Wo."""
    OA = _as(nested_output_matrix(g.base, g.lv), exact)
    Mn = g.lv.Mn
    dt = object if exact else np.float64
    y = np.zeros((g.B, g.N, g.th * Mn, g.tw * Mn), dtype=dt)
    for b in range(g.B):
        for ty in range(g.th):
            for tx in range(g.tw):
                for n in range(g.N):
                    y[b, n, ty * Mn:(ty + 1) * Mn, tx * Mn:(tx + 1) * Mn] = \
                        OA.dot(Yh[b, ty, tx, n].dot(OA.T))
    return y[:, :, :g.Ho, :g.Wo]


def _to_fractions(a) -> np.ndarray:
    a = np.asarray(a)
    out = np.empty(a.shape, dtype=object)
    for idx in np.ndindex(a.shape):
        out[idx] = Fraction(a[idx]) if not isinstance(a[idx], Fraction) else a[idx]
    return out


def nested_conv2d(x, w, pad: int = 0, base: Optional[Base] = None, exact: bool = False,
                  counter: Optional[MultCounter] = None) -> np.ndarray:
    """Stride-1 2D correlation by nested Winograd (steps 1-6 of the module doc).

    ``exact=True`` runs in rational arithmetic (inputs converted to Fraction);
    otherwise fp64.  Returns y[B][N][Ho][Wo].
    """
    g = geometry(np.shape(x), np.shape(w), pad, base)
    if exact:
        x, w = _to_fractions(x), _to_fractions(w)
    if g.lv.n == 0:
        # F(1, r): no overlap between tiles, the native convolution (1x1 kernel).
        ws = w if exact else np.asarray(w, np.float64)
        xp = padded_input(x, g, exact)
        y = np.zeros((g.B, g.N, g.Ho, g.Wo), dtype=object if exact else np.float64)
        if exact:
            y[:] = Fraction(0)
        for b in range(g.B):
            for n in range(g.N):
                for m in range(g.M):
                    y[b, n] = y[b, n] + ws[n, m, 0, 0] * xp[b, m, :g.Ho, :g.Wo]
        if counter is not None:
            counter.count += g.B * g.N * g.M * g.Ho * g.Wo
        return y
    U = kernel_transform(w, g, exact)
    V = input_transform(x, g, exact)
    Yh = ewmm(U, V, counter)
    return output_transform(Yh, g, exact)


def depthwise_geometries(x_shape, w_shape, pad: int, base: Optional[Base] = None):
    """(kernel geometry, data geometry) of a depthwise layer x [B][C][H][W], w [C][1][r][r].

    The kernel transform sees C kernels of one input channel (N = C, M = 1);
    the input and output transforms see C channels (M = N = C).
    """
    B, C, H, W = x_shape
    Cw, one, r, r2 = w_shape
    if Cw != C or one != 1 or r != r2:
        raise ValueError("x must be [B][C][H][W] and w [C][1][r][r]")
    return (geometry((B, 1, H, W), w_shape, pad, base),
            geometry(x_shape, (C, C, r, r), pad, base))


def nested_depthwise_conv2d(x, w, pad: int = 0, base: Optional[Base] = None,
                            exact: bool = False,
                            counter: Optional[MultCounter] = None) -> np.ndarray:
    """Depthwise correlation by nested Winograd: the same transforms as
    nested_conv2d, with the element-wise product of each channel's own
    transformed kernel and no sum over channels."""
    gk, gx = depthwise_geometries(np.shape(x), np.shape(w), pad, base)
    if exact:
        x, w = _to_fractions(x), _to_fractions(w)
    if gx.lv.n == 0:
        # 1x1 kernel: each channel scaled by its single weight
        ws = w if exact else np.asarray(w, np.float64)
        xp = padded_input(x, gx, exact)
        if counter is not None:
            counter.count += gx.B * gx.N * gx.Ho * gx.Wo
        return ws[None, :, 0, 0:1, 0:1] * xp[:, :, :gx.Ho, :gx.Wo]
    U = kernel_transform(w, gk, exact)
    V = input_transform(x, gx, exact)
    Yh = ewmm_depthwise(U, V, counter)
    return output_transform(Yh, gx, exact)
