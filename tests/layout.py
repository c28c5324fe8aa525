"""The library's Winograd-domain buffer layouts, built from the CPU oracle's
arrays (test helpers; no device work).

The library orders a tile's P points by the base-4 digits (q_n^row, q_n^col,
..., q_1^row, q_1^col), most significant first, and stores Winograd-domain
buffers quad-interleaved ([P/4][X][Y][4], the level-1 column digit
innermost).  Z is the contraction's output after the level-1 output
transform.
"""
import numpy as np

from oracle.nested import base_f23, point_permutation


def to_lib_points(a, n):
    """oracle [..., P1, P1] -> [..., P] in the library's point order."""
    perm = point_permutation(n)
    return a[..., perm[:, 0], perm[:, 1]]


def quads(a_pxy):
    """[P][X][Y] -> quad-interleaved [P/4][X][Y][4]."""
    P, X, Y = a_pxy.shape
    return np.ascontiguousarray(a_pxy.reshape(P // 4, 4, X, Y).transpose(0, 2, 3, 1))


def level1(yh_pnt):
    """[P][N][T] -> Z [P/16][N][T][4]: the oracle's A^T along both level-1 digits."""
    AT = base_f23().AT.astype(np.float64)
    P, N, T = yh_pnt.shape
    g = yh_pnt.reshape(P // 16, 4, 4, N, T)
    z = np.einsum("iq,jr,gqrnt->gntij", AT, AT, g)
    return np.ascontiguousarray(z.reshape(P // 16, N, T, 4))
