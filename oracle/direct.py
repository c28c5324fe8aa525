"""Direct stride-1 2D convolution in fp64 -- the oracle's plain definition.

Test infrastructure only (see ``oracle/__init__.py``).

Sec. II.A: M input maps x of size HxW are correlated with N groups of
M-channel kernels w of size RxR (here R = r) to give N output maps y; the
window slides by 1.  With zero padding p on all four sides:

    y[b,n,i,j] = sum_{m<M} sum_{u<r} sum_{v<r} xp[b,m,i+u,j+v] * w[n,m,u,v]

for 0 <= i < Ho = H + 2p - r + 1 and 0 <= j < Wo = W + 2p - r + 1, where xp
is x zero-padded by p.  There is no kernel flip: the paper describes the
operation as a correlation, and the base matrices of eq. 2.3 compute one.
"""
from __future__ import annotations

import numpy as np


def _check(x, w, pad):
    if x.ndim != 4 or w.ndim != 4:
        raise ValueError("x must be [B][M][H][W] and w [N][M][r][r]")
    B, M, H, W = x.shape
    N, Mw, r, r2 = w.shape
    if Mw != M or r != r2:
        raise ValueError("channel count or kernel shape mismatch")
    Ho, Wo = H + 2 * pad - r + 1, W + 2 * pad - r + 1
    if Ho <= 0 or Wo <= 0:
        raise ValueError("kernel larger than the padded input")
    return B, M, H, W, N, r, Ho, Wo


def direct_conv2d(x, w, pad: int = 0) -> np.ndarray:
    """fp64 direct correlation, computed as r*r shifted GEMMs.

    For each kernel tap (u, v) the shifted input window is an (M x B*Ho*Wo)
    matrix; w[:, :, u, v] (N x M) times it is that tap's contribution to
    every output.  Returns y[B][N][Ho][Wo] in float64.
    """
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    B, M, H, W, N, r, Ho, Wo = _check(x, w, pad)
    xp = np.pad(x, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    xpt = xp.transpose(1, 0, 2, 3)            # [M][B][Hp][Wp]
    # taps outermost, so that each tap's N x M matrix is contiguous and the
    # product goes to BLAS (numpy multiplies a strided view with its own loop)
    wt = np.ascontiguousarray(w.transpose(2, 3, 0, 1))   # [r][r][N][M]
    y = np.zeros((N, B * Ho * Wo), dtype=np.float64)
    for u in range(r):
        for v in range(r):
            win = np.ascontiguousarray(xpt[:, :, u:u + Ho, v:v + Wo]).reshape(M, -1)
            y += wt[u, v] @ win
    return y.reshape(N, B, Ho, Wo).transpose(1, 0, 2, 3).copy()


def brute_force_conv2d(x, w, pad: int = 0) -> np.ndarray:
    """The same definition as nested Python loops over every index.

    Only for tiny inputs; it exists to pin ``direct_conv2d``.
    """
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    B, M, H, W, N, r, Ho, Wo = _check(x, w, pad)
    y = np.zeros((B, N, Ho, Wo), dtype=np.float64)
    for b in range(B):
        for n in range(N):
            for i in range(Ho):
                for j in range(Wo):
                    acc = 0.0
                    for m in range(M):
                        for u in range(r):
                            for v in range(r):
                                ii, jj = i + u - pad, j + v - pad
                                if 0 <= ii < H and 0 <= jj < W:
                                    acc += float(x[b, m, ii, jj]) * float(w[n, m, u, v])
                    y[b, n, i, j] = acc
    return y


def direct_depthwise_conv2d(x, w, pad: int = 0) -> np.ndarray:
    """fp64 depthwise correlation: one r x r kernel per channel, no channel sum.

    Table I's depth-wise row: x [B][C][H][W], w [C][1][r][r],

        y[b,c,i,j] = sum_{u<r} sum_{v<r} xp[b,c,i+u,j+v] * w[c,0,u,v],

    computed as r*r shifted windows, each scaled per channel.
    """
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    if x.ndim != 4 or w.ndim != 4 or w.shape[1] != 1 or w.shape[0] != x.shape[1] \
            or w.shape[2] != w.shape[3]:
        raise ValueError("x must be [B][C][H][W] and w [C][1][r][r]")
    B, C, H, W = x.shape
    r = w.shape[2]
    Ho, Wo = H + 2 * pad - r + 1, W + 2 * pad - r + 1
    if Ho <= 0 or Wo <= 0:
        raise ValueError("kernel larger than the padded input")
    xp = np.pad(x, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    y = np.zeros((B, C, Ho, Wo), dtype=np.float64)
    for u in range(r):
        for v in range(r):
            y += w[None, :, 0, u, v, None, None] * xp[:, :, u:u + Ho, v:v + Wo]
    return y


def direct_conv2d_points(x, w, pad: int, points) -> np.ndarray:
    """Selected outputs y[b,n,i,j] of the same definition, one at a time.

    ``points`` is an iterable of (b, n, i, j).  Used to check full-size GPU
    results on a sample of outputs without computing the whole convolution.
    """
    x = np.asarray(x)
    w = np.asarray(w)
    B, M, H, W, N, r, Ho, Wo = _check(x, w, pad)
    out = []
    for (b, n, i, j) in points:
        i0, j0 = i - pad, j - pad
        u0, v0 = max(0, -i0), max(0, -j0)
        u1, v1 = min(r, H - i0), min(r, W - j0)
        patch = x[b, :, i0 + u0:i0 + u1, j0 + v0:j0 + v1].astype(np.float64)
        ker = w[n, :, u0:u1, v0:v1].astype(np.float64)
        out.append(float(np.sum(patch * ker)))
    return np.asarray(out, dtype=np.float64)
