"""GPU parity of the mixed nest (NWG_TILE_MIX_F23_F33: F(2,3) at levels 1-2,
F(3,3) above; depth 3 for r = 8..15, depth 4 for r = 16..39) against the CPU
oracle.

End to end against the fp64 direct convolution (rel-L2 <= 1e-4, max-abs <=
1e-3 max|y|); stage by stage against the oracle's mixed-chain transforms
(oracle/mixed.py: input, kernel and output matrices of the chain), re-ordered
to the library's mixed-radix point order.  Inputs are seeded and synthetic.
"""
import numpy as np
import pytest
import torch

from oracle.direct import direct_conv2d
from oracle.mixed import input_matrix, kernel_matrix, mixed_levels, output_matrix
from oracle.nested import ewmm
from paper_2102_13272_amd import nwg
from paper_2102_13272_amd.workloads import make_case
from tests.gpu_util import assert_close, dev
from tests.layout import (level1, live_group_mask, mixed_chain, mixed_to_lib_points,
                          planar_group_index, planar_points, quads)

pytestmark = pytest.mark.gpu
MIX = nwg.NWG_TILE_MIX_F23_F33


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nwg.load_library()          # raises if the HIP library is missing: no fallback


def _conv(x, w, pad):
    B, M, H, W = x.shape
    N, _, r, _ = w.shape
    with nwg.Plan(B, M, N, H, W, r, pad, tile=MIX) as plan:
        i = plan.info
        assert i["tile"] == MIX and i["outer33"] == i["n"] - 2
        assert i["fused_input"] == i["fused_conv"] == i["fused_output"] == 0
        y = torch.full(plan.y_shape, float("nan"), device="cuda")
        plan.conv2d(dev(x), dev(w), y)
        torch.cuda.synchronize()
        return y.cpu().numpy().astype(np.float64)


# B, M, N, H, W, r, pad: depth 3 (M_n = 12) and 4 (M_n = 36), ragged tiles,
# one tile, odd channel counts, one channel, the deep contraction (M % 32,
# N % 64, T = 64) plain and persistent (depth 4: 10000 groups), r = 39
E2E = [
    (1, 3, 5, 30, 27, 8, 3),
    (2, 5, 4, 41, 29, 13, 6),
    (1, 4, 3, 26, 26, 15, 0),
    (1, 1, 1, 20, 20, 9, 4),
    (16, 32, 64, 24, 24, 13, 6),
    (1, 3, 2, 60, 50, 16, 7),
    (1, 2, 3, 75, 40, 31, 15),
    (1, 2, 2, 45, 45, 39, 19),
    (2, 33, 20, 40, 40, 23, 11),
    (3, 4, 5, 37, 50, 20, 0),       # no padding, rectangular, B = 3
    (1, 6, 7, 90, 30, 12, 5),       # depth 3, a tall image (8 x 3 tiles)
    (1, 65, 17, 40, 40, 16, 8),     # M = 65, N = 17: ragged kernel-transform blocks
    (10, 2, 3, 72, 72, 31, 15),     # depth 4, T = 40: a full 32-tile input chunk and a ragged one
]


@pytest.mark.parametrize("case", E2E, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_mixed_conv2d_matches_direct_oracle(case):
    B, M, N, H, W, r, pad = case
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=7 * sum(case))
    print(f"mixed case {case}", flush=True)
    assert_close(_conv(x, w, pad), direct_conv2d(x, w, pad), what=str(case))


# the deep contraction at depth 4 (T = 64, 10000 groups: the persistent
# form), 64 x 64 blocks (N = 64) and 128 x 64 blocks (N = 128), compared
# output by output
BIG = [(64, 32, 64, 36, 36, 31, 15), (64, 32, 128, 36, 36, 31, 15)]


@pytest.mark.parametrize("case", BIG, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_mixed_conv2d_deep_contraction_whole_output(case):
    B, M, N, H, W, r, pad = case
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=7 * sum(case))
    print(f"mixed case {case}", flush=True)
    with nwg.Plan(B, M, N, H, W, r, pad, tile=MIX) as plan:
        assert (plan.info["n"], plan.info["T"]) == (4, 64)
    assert_close(_conv(x, w, pad), direct_conv2d(x, w, pad), what=str(case))


def _stage_refs(x, w, pad):
    """The oracle chain's U, V, Yhat per tile and y (as in nested_conv2d_mixed),
    from its input, kernel and output matrices."""
    B, M, H, W = x.shape
    N, _, r, _ = w.shape
    lv = mixed_levels(mixed_chain(), r)
    Mn, Ln, P1 = lv.Mn, lv.Ln, lv.P1
    IB, KG, OA = (np.asarray(m, dtype=np.float64)
                  for m in (input_matrix(lv), kernel_matrix(lv), output_matrix(lv)))
    Ho, Wo = H + 2 * pad - r + 1, W + 2 * pad - r + 1
    th, tw = -(-Ho // Mn), -(-Wo // Mn)
    wp = np.zeros((N, M, lv.Kn, lv.Kn))
    wp[:, :, :r, :r] = w
    U = np.einsum("pk,nmkl,ql->nmpq", KG, wp, KG, optimize=True)
    Hp, Wp = (th - 1) * Mn + Ln, (tw - 1) * Mn + Ln
    xp = np.zeros((B, M, max(Hp, H + pad), max(Wp, W + pad)))
    xp[:, :, pad:pad + H, pad:pad + W] = x
    V = np.empty((B, th, tw, M, P1, P1))
    for ty in range(th):
        for tx in range(tw):
            X = xp[:, :, ty * Mn:ty * Mn + Ln, tx * Mn:tx * Mn + Ln]
            V[:, ty, tx] = np.einsum("pk,bmkl,ql->bmpq", IB, X, IB, optimize=True)
    Yh = ewmm(U, V)
    y = np.zeros((B, N, th * Mn, tw * Mn))
    for ty in range(th):
        for tx in range(tw):
            y[:, :, ty * Mn:(ty + 1) * Mn, tx * Mn:(tx + 1) * Mn] = \
                np.einsum("ip,bnpq,jq->bnij", OA, Yh[:, ty, tx], OA, optimize=True)
    return lv, U, V, Yh, y[:, :, :Ho, :Wo]


STAGES = [(1, 3, 4, 30, 28, 13, 6), (2, 2, 3, 20, 22, 8, 0), (1, 2, 3, 40, 38, 20, 9)]


@pytest.mark.parametrize("case", STAGES, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_mixed_stages_match_cpu_oracle_chain(case):
    B, M, N, H, W, r, pad = case
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=11 + r)
    print(f"mixed stages {case}", flush=True)
    lv, U_ref, V_ref, Yh_ref, y_ref = _stage_refs(x, w, pad)
    radices = [b.l for b in lv.bases]
    P1 = lv.P1
    T = V_ref.shape[0] * V_ref.shape[1] * V_ref.shape[2]
    U_lib = np.ascontiguousarray(mixed_to_lib_points(U_ref, radices).transpose(2, 1, 0))
    V_lib = np.ascontiguousarray(
        mixed_to_lib_points(V_ref.reshape(T, M, P1, P1), radices).transpose(2, 1, 0))
    Yh_lib = mixed_to_lib_points(Yh_ref.reshape(T, N, P1, P1), radices).transpose(2, 1, 0)
    Z_lib = level1(Yh_lib)
    # the oracle chain itself equals the direct convolution (pinned in the CPU suite)
    assert_close(y_ref, direct_conv2d(x, w, pad), rel_tol=1e-9, abs_frac=1e-9, what="oracle")

    with nwg.Plan(B, M, N, H, W, r, pad, tile=MIX) as plan:
        i = plan.info
        assert (i["n"], i["P"], i["T"], i["Mn"]) == (lv.n, P1 * P1, T, lv.Mn)
        assert i["yhat_bytes"] == 4 * Z_lib.size and i["v_bytes"] == 4 * V_lib.size
        U = torch.full(plan.u_shape, float("nan"), device="cuda")
        V = torch.full(plan.v_shape, float("nan"), device="cuda")
        Z = torch.full(plan.z_shape, float("nan"), device="cuda")
        y = torch.full(plan.y_shape, float("nan"), device="cuda")
        # the live groups: the dead ones' oracle U and Z are exactly zero, and
        # the library neither writes nor reads their U, V and Z
        live = live_group_mask(i)
        lq = np.repeat(live, 4)                     # a group is 4 quads of U and V
        if i["level1_live"] == 0x7:                 # level-1 digit 3 dead: quads q1r = 3 too
            lq &= np.arange(lq.size) % 4 != 3
        assert live.sum() == (i["live_groups"] if i["live_np"] else i["P"] // 16)
        assert not np.any(quads(U_lib)[~lq]) and not np.any(Z_lib[~live])
        if i["level1_live"] == 0x7:                 # and the q1c = 3 lane of every quad
            assert not np.any(quads(U_lib)[..., 3])
        plan.kernel_transform(dev(w), U)
        plan.input_transform(dev(x), V)
        torch.cuda.synchronize()
        # fp32 rounding of B^T's thirds and sixths and G's 4s over the levels
        # the live lanes (q1c = 3 is a dead point too when digit 3 is dead)
        nl = 3 if i["level1_live"] == 0x7 else 4
        assert_close(U.cpu().numpy()[lq][..., :nl], quads(U_lib)[lq][..., :nl],
                     rel_tol=1e-6, abs_frac=1e-6, what="U")
        assert_close(V.cpu().numpy()[lq][..., :nl], quads(V_lib)[lq][..., :nl],
                     rel_tol=1e-6, abs_frac=1e-6, what="V")
        Vq = quads(V_lib)
        Vq[~lq] = np.nan                            # never read
        plan.contract(dev(quads(U_lib)), dev(Vq), Z)
        torch.cuda.synchronize()
        Zg = Z.cpu().numpy()
        assert_close(Zg[live], Z_lib[live], rel_tol=1e-5, abs_frac=1e-5, what="Z")
        assert np.isnan(Zg[~live]).all()            # not written
        Z_lib = Z_lib.copy()
        Z_lib[~live] = np.nan                       # never read
        plan.output_transform(dev(Z_lib), y)
        torch.cuda.synchronize()
        # fp32 sums over A^T entries up to 4 at the F(3,3) levels (rows and
        # columns, two levels at depth 4): ~1e-6 of the output's norm
        assert_close(y.cpu().numpy(), y_ref, rel_tol=1e-5, abs_frac=1e-5, what="y")


# the planar layout (mix_planar: depth 4, level-1 digit 3 dead, M % 128,
# N % 128, T % 64): one 36 x 36 tile per image, T = 64 or 128, 128 x 64
# blocks in one or two rows, r = 23 to 35, 128 or 256 input channels
PLANAR = [(64, 128, 128, 36, 36, 31, 15), (64, 128, 256, 36, 36, 31, 15),
          (128, 128, 128, 36, 36, 23, 11), (16, 128, 128, 72, 72, 27, 13),
          (64, 128, 128, 36, 36, 35, 17), (64, 256, 128, 36, 36, 31, 15)]


@pytest.mark.parametrize("case", PLANAR, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_mixed_planar_conv2d_sampled_outputs(case):
    """Whole layers on the planar layout against the direct oracle on sampled
    images and output channels (every output position of those)."""
    B, M, N, H, W, r, pad = case
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=3 * sum(case))
    print(f"mixed planar case {case}", flush=True)
    with nwg.Plan(B, M, N, H, W, r, pad, tile=MIX) as plan:
        assert plan.info["mix_planar"] == 1
    y = _conv(x, w, pad)
    bs = sorted({0, B // 2, B - 1})
    ns = sorted({0, 1, N // 2 + 3, N - 1})
    ref = direct_conv2d(x[bs], w[ns], pad)
    assert_close(y[np.ix_(bs, ns)], ref, what=str(case))


def test_mixed_planar_stages_sampled():
    """Stage by stage on the planar layout: U and V at sampled (channel, tile)
    against the oracle's kernel and input matrices at every live point; the
    contraction on seeded random U and V against an fp64 sum on sampled
    groups, the dead groups' Z untouched."""
    B, M, N, H, W, r, pad = PLANAR[0]
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=5)
    print(f"mixed planar stages {PLANAR[0]}", flush=True)
    lv = mixed_levels(mixed_chain(), r)
    KG = np.asarray(kernel_matrix(lv), dtype=np.float64)
    IB = np.asarray(input_matrix(lv), dtype=np.float64)
    with nwg.Plan(B, M, N, H, W, r, pad, tile=MIX) as plan:
        i = plan.info
        G = i["live_groups"]
        assert i["mix_planar"] == 1 and (i["T"], i["th"], i["tw"]) == (B, 1, 1)
        assert plan.u_shape == (G, 9, M, N) and plan.v_shape == (G, 9, M, B)
        rows, cols = planar_points(i)
        U = torch.full(plan.u_shape, float("nan"), device="cuda")
        V = torch.full(plan.v_shape, float("nan"), device="cuda")
        plan.kernel_transform(dev(w), U)
        plan.input_transform(dev(x), V)
        torch.cuda.synchronize()
        Uh, Vh = U.cpu().numpy(), V.cpu().numpy()
        del U, V
        for n, m in [(0, 0), (N - 1, M - 1), (37, 101)]:
            wp = np.zeros((lv.Kn, lv.Kn))
            wp[:r, :r] = w[n, m]
            Uo = KG @ wp @ KG.T
            assert_close(Uh[:, :, m, n], Uo[rows, cols], rel_tol=1e-6, abs_frac=1e-6,
                         what=f"U n={n} m={m}")
        for b, m in [(0, 0), (B - 1, M - 1), (20, 77)]:
            X = np.zeros((lv.Ln, lv.Ln))
            X[pad:pad + H, pad:pad + W] = x[b, m, :lv.Ln - pad, :lv.Ln - pad]
            Vo = IB @ X @ IB.T
            assert_close(Vh[:, :, m, b], Vo[rows, cols], rel_tol=1e-6, abs_frac=1e-6,
                         what=f"V b={b} m={m}")
        del Uh, Vh
        rng = np.random.default_rng(3)
        Ur = rng.standard_normal(plan.u_shape, dtype=np.float32)
        Vr = rng.standard_normal(plan.v_shape, dtype=np.float32)
        Z = torch.full(plan.z_shape, float("nan"), device="cuda")
        plan.contract(dev(Ur), dev(Vr), Z)
        torch.cuda.synchronize()
        Zh = Z.cpu().numpy()
    assert np.isnan(Zh[~live_group_mask(i)]).all()     # dead groups: not written
    AT = np.array([[1.0, 1.0, 1.0], [0.0, 1.0, -1.0]])  # A^T of F(2,3) on digits 0..2
    for li in [0, 1, 1234, G // 2, G - 1]:
        prod = np.einsum("pmn,pmt->pnt", Ur[li].astype(np.float64), Vr[li].astype(np.float64))
        zr = np.zeros((N, B, 4))
        for p in range(9):
            q1r, q1c = divmod(p, 3)
            for i1r in range(2):
                for i1c in range(2):
                    zr[..., 2 * i1r + i1c] += AT[i1r, q1r] * AT[i1c, q1c] * prod[p]
        assert_close(Zh[planar_group_index(i, li)], zr, rel_tol=1e-5, abs_frac=1e-5,
                     what=f"Z group {li}")


@pytest.mark.parametrize("r,N", [(17, 128), (31, 256), (32, 128), (35, 128), (38, 128)])
def test_mixed_planar_kernel_transform_matches_oracle(r, N):
    """The planar kernel transform at both of its work-group widths (32
    output channels when their kernels fit in LDS, r <= 31; 16 above): every
    place of U written, and U at every live point for sampled (n, m) against
    the oracle's kernel matrix."""
    B, M, H = 64, 128, 36
    pad = (r - 1) // 2
    rng = np.random.default_rng(r * 1000 + N)
    w = (rng.standard_normal((N, M, r, r)) / np.sqrt(M * r * r)).astype(np.float32)
    lv = mixed_levels(mixed_chain(), r)
    KG = np.asarray(kernel_matrix(lv), dtype=np.float64)
    print(f"mixed planar kernel transform r={r} N={N}", flush=True)
    with nwg.Plan(B, M, N, H, H, r, pad, tile=MIX) as plan:
        i = plan.info
        assert i["mix_planar"] == 1
        rows, cols = planar_points(i)
        U = torch.full(plan.u_shape, float("nan"), device="cuda")
        plan.kernel_transform(dev(w), U)
        torch.cuda.synchronize()
        Uh = U.cpu().numpy()
        del U
    assert np.isfinite(Uh).all()
    for n, m in [(0, 0), (N - 1, M - 1), (31, 5), (32, 77), (N // 2 + 15, 64)]:
        wp = np.zeros((lv.Kn, lv.Kn))
        wp[:r, :r] = w[n, m]
        Uo = KG @ wp @ KG.T
        assert_close(Uh[:, :, m, n], Uo[rows, cols], rel_tol=1e-6, abs_frac=1e-6,
                     what=f"U r={r} n={n} m={m}")


def test_mixed_plan_rejects_what_it_does_not_serve():
    with pytest.raises(nwg.NwgError):
        nwg.Plan(1, 2, 2, 90, 90, 40, 0, tile=MIX)                 # r > 39
    with pytest.raises(nwg.NwgError):
        nwg.Plan(1, 2, 2, 40, 40, 9, 4, tile=MIX, depthwise=True)
    with nwg.Plan(1, 3, 1, 40, 40, 13, 6, tile=MIX) as plan:
        assert plan.info["fused_input"] == 0
        U = torch.empty(plan.u_shape, device="cuda")
        Z = torch.empty(plan.z_shape, device="cuda")
        x = torch.zeros((1, 3, 40, 40), device="cuda")
        with pytest.raises(nwg.NwgError):
            plan.input_contract(x, U, Z)
        with pytest.raises(nwg.NwgError):
            plan.set_pipeline(2)
        with pytest.raises(nwg.NwgError):
            plan.set_precision(nwg.NWG_PRECISION_BF16_SPLIT)
    # r <= 7: the F(2x2,3x3) plan
    with nwg.Plan(1, 2, 2, 30, 30, 7, 3, tile=MIX) as plan:
        assert plan.info["tile"] == nwg.NWG_TILE_F2X2_3X3


def test_large_kernel_workload_on_the_mixed_nest_at_tile_edges(c5_oracle):
    """The 31x31 workload on the mixed nest (n = 4, 36 x 36 tiles, the second
    ragged), whole output against the oracle, and on its own the outputs on
    both sides of the 12-pixel level-3 blocks and the 36-pixel tile edge."""
    L, x, w, ref = c5_oracle
    print("workload c5_r31 mixed nest", flush=True)
    with nwg.Plan(L.B, L.M, L.N, L.H, L.W, L.r, L.pad, tile=MIX) as plan:
        assert (plan.info["n"], plan.info["Mn"], plan.info["T"]) == (4, 36, 64)
        y = torch.empty(plan.y_shape, device="cuda")
        plan.conv2d(dev(x), dev(w), y)
        torch.cuda.synchronize()
        yh = y.cpu().numpy()
    assert np.isfinite(yh).all()
    assert_close(yh, ref, what="c5_r31 mixed")
    edges = [0, 11, 12, 23, 24, 35, 36, 47, 48, L.Ho - 1]
    sub = np.ix_(range(L.B), range(L.N), edges, edges)
    assert_close(yh[sub], ref[sub], what="tile and block edges")
