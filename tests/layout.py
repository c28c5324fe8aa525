"""The library's Winograd-domain buffer layouts, built from the CPU oracle's
arrays (test helpers; no device work).

The library orders a tile's P points by the base-4 digits (q_n^row, q_n^col,
..., q_1^row, q_1^col), most significant first, and stores Winograd-domain
buffers quad-interleaved ([P/4][X][Y][4], the level-1 column digit
innermost).  Z is the contraction's output after the level-1 output
transform.
"""
import numpy as np

from oracle.nested import base_f23, toom_cook_base


def point_permutation(n: int, l: int = 4) -> np.ndarray:
    """Map the library's flat point index p to the oracle's (row, column) point.

    The library orders the P = l^(2n) points of a tile by the base-l digits
    (q_n^row, q_n^col, q_{n-1}^row, q_{n-1}^col, ..., q_1^row, q_1^col), most
    significant first, where q_j is the level-j index.  The oracle indexes a
    point as [pi_row, pi_col] with pi = (q_1, ..., q_n), q_1 most significant.
    Returns an int array perm of shape (P, 2) with perm[p] = (pi_row, pi_col).
    """
    P = l ** (2 * n)
    perm = np.zeros((P, 2), dtype=np.int64)
    for p in range(P):
        digits = []
        rem = p
        for _ in range(2 * n):
            digits.append(rem % l)
            rem //= l
        digits = digits[::-1]       # most significant first
        q_row = {n - k: digits[2 * k] for k in range(n)}      # level index -> digit
        q_col = {n - k: digits[2 * k + 1] for k in range(n)}
        pr = 0
        pc = 0
        for j in range(1, n + 1):   # q_1 most significant in the oracle
            pr = pr * l + q_row[j]
            pc = pc * l + q_col[j]
        perm[p] = (pr, pc)
    return perm


def to_lib_points(a, n, l=4):
    """oracle [..., P1, P1] -> [..., P] in the library's point order (base-l
    digits)."""
    perm = point_permutation(n, l)
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


def f33_base():
    """F(3,3) from the Toom-Cook points 0, 1, -1, 2 (and infinity), the base of
    the library's F(3x3, 3x3) tile."""
    return toom_cook_base(3, 3, [0, 1, -1, 2])


def level1_f33(yh_pnt):
    """F(3,3) tile: [P][N][T] -> Z [P/25][5][3][N][T] with
    Z[g][q1r][i1c] = sum_{q1c} A^T[i1c][q1c] Yhat[25 g + 5 q1r + q1c] (the
    oracle's A^T along the level-1 columns only)."""
    AT = f33_base().AT.astype(np.float64)
    P, N, T = yh_pnt.shape
    g = yh_pnt.reshape(P // 25, 5, 5, N, T)
    return np.ascontiguousarray(np.einsum("jr,gqrnt->gqjnt", AT, g))


def mixed_chain():
    """The library's mixed nest: F(2,3) at levels 1 and 2, F(3,3) above."""
    f23, f33 = base_f23(), f33_base()
    return [f23, f23, f33, f33]


def mixed_to_lib_points(a, radices):
    """oracle [..., P1, P1] of a mixed chain (per-axis index with level 1 most
    significant, radices l_1..l_n) -> [..., P] in the library's order: digits
    (q_n^row, q_n^col, ..., q_1^row, q_1^col), most significant first."""
    n = len(radices)
    shape = []
    for j in range(n - 1, -1, -1):
        shape += [radices[j], radices[j]]
    idx = np.indices(shape).reshape(2 * n, -1)      # lib digits, most significant first
    rows = np.zeros(idx.shape[1], dtype=np.int64)
    cols = np.zeros(idx.shape[1], dtype=np.int64)
    for j in range(n):                              # level j + 1, most significant first
        k = 2 * (n - 1 - j)
        rows = rows * radices[j] + idx[k]
        cols = cols * radices[j] + idx[k + 1]
    return a[..., rows, cols]


def live_group_mask(info):
    """Per group (P/16, the library's order) whether it is live for the plan
    (nwg_plan_info live_np, live_prefix): its row prefix (q_n^r .. q_2^r) and
    its column prefix are both live.  A prefix's bit index has q_2 least
    significant (radix 4), then q_3, ... (radix 5 on the mixed nest, 4 on a
    chain of F(2x2,3x3) levels).  Every group when live_np is 0."""
    from paper_2102_13272_amd import nwg
    G = info["P"] // 16
    if info["live_np"] == 0:
        return np.ones(G, dtype=bool)
    mask = int(info["live_prefix"][0]) | (int(info["live_prefix"][1]) << 64)
    up = 5 if info["tile"] == nwg.NWG_TILE_MIX_F23_F33 else 4
    radix = [4] + [up] * (info["n"] - 2)            # levels 2 .. n
    out = np.empty(G, dtype=bool)
    for g in range(G):
        rest, pr, pc, mul = g, 0, 0, 1
        for l in radix:                             # group digits (row, col) per level, q_2 last
            pc += (rest % l) * mul
            rest //= l
            pr += (rest % l) * mul
            rest //= l
            mul *= l
        out[g] = bool((mask >> pr) & 1) and bool((mask >> pc) & 1)
    return out


def live_prefixes(info):
    """The live axis prefixes of a mixed plan, in prefix order (bit i of
    live_prefix: i = (q_4 * 5 + q_3) * 4 + q_2 at depth 4)."""
    mask = int(info["live_prefix"][0]) | (int(info["live_prefix"][1]) << 64)
    return [i for i in range(128) if (mask >> i) & 1]


def mixed_axis_index(q1, prefix):
    """Depth-4 mixed nest: the oracle's per-axis point index (level 1 most
    significant, radices 4, 4, 5, 5) of level-1 digit q1 under axis prefix
    (q_4 * 5 + q_3) * 4 + q_2."""
    q2, q3, q4 = prefix % 4, (prefix // 4) % 5, prefix // 20
    return ((q1 * 4 + q2) * 5 + q3) * 5 + q4


def planar_points(info):
    """Row and column oracle axis indices [live_groups][9] of the planar
    layout's points: group i = (row rank, column rank) = divmod(i, live_np),
    point p = 3 q1r + q1c."""
    pre = live_prefixes(info)
    np_ = info["live_np"]
    rows = np.empty((np_ * np_, 9), dtype=np.int64)
    cols = np.empty_like(rows)
    for i in range(np_ * np_):
        pr, pc = pre[i // np_], pre[i % np_]
        for p in range(9):
            rows[i, p] = mixed_axis_index(p // 3, pr)
            cols[i, p] = mixed_axis_index(p % 3, pc)
    return rows, cols


def planar_group_index(info, i):
    """Z's group index g of the planar layout's group i."""
    pre = live_prefixes(info)
    np_ = info["live_np"]
    pr, pc = pre[i // np_], pre[i % np_]
    g = 0
    for d, (wr, wc) in enumerate([(4, 1), (80, 16), (2000, 400)]):   # q_2, q_3, q_4
        rad = 4 if d == 0 else 5
        g += (pr % rad) * wr + (pc % rad) * wc
        pr //= rad
        pc //= rad
    return g
