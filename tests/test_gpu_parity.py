"""GPU parity of the HIP nested-Winograd path against the CPU oracle.

End to end: y from nwg_conv2d against the fp64 direct convolution
(rel-L2 <= 1e-4, max-abs <= 1e-3 max|y|).  Stage by stage: the library's
U, V, Yhat against the CPU nested reference, re-ordered to the library's
documented point order.  All inputs are seeded and synthetic.
"""
import numpy as np
import pytest
import torch

from oracle.direct import direct_conv2d
from oracle.nested import ewmm, geometry, input_transform, kernel_transform, output_transform
from paper_2102_13272_amd import nwg
from paper_2102_13272_amd.workloads import make_case
from tests.gpu_util import assert_close, dev, run_conv
from tests.layout import (level1 as _level1, live_group_mask, quads as _quads,
                          to_lib_points as _to_lib_points)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nwg.load_library()          # raises if the HIP library is missing: no fallback


# B, M, N, H, W, r, pad -- depths 0..4, ragged tiles, odd channel counts, B > 1
E2E = [
    (2, 3, 5, 9, 7, 1, 0),
    (1, 4, 4, 16, 16, 4, 0),
    (1, 5, 3, 11, 13, 2, 0),
    (2, 5, 5, 19, 17, 3, 1),
    (1, 1, 7, 23, 21, 5, 2),
    (3, 6, 4, 17, 30, 7, 3),
    (1, 9, 1, 21, 18, 9, 4),
    (2, 7, 9, 29, 26, 13, 6),
    (1, 3, 2, 15, 15, 15, 0),
    (1, 2, 3, 40, 35, 31, 15),
    (1, 17, 20, 31, 31, 31, 0),   # a single output pixel
    (1, 33, 18, 24, 24, 16, 0),
]


@pytest.mark.parametrize("case", E2E, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_conv2d_matches_direct_oracle(case):
    B, M, N, H, W, r, pad = case
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=sum(case))
    print(f"case {case}", flush=True)
    y = run_conv(x, w, pad)
    assert_close(y, direct_conv2d(x, w, pad), what=str(case))


STAGES = [(1, 3, 4, 12, 10, 3, 1), (2, 4, 3, 13, 11, 6, 2), (1, 3, 5, 20, 19, 11, 5),
          (1, 2, 3, 24, 20, 31, 15), (2, 5, 2, 9, 9, 2, 0)]


@pytest.mark.parametrize("case", STAGES, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_stages_match_cpu_nested_reference(case):
    B, M, N, H, W, r, pad = case
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=7 + r)
    print(f"stages {case}", flush=True)
    g = geometry(x.shape, w.shape, pad)
    n = g.lv.n
    U_ref = kernel_transform(w, g)                      # (N, M, P1, P1)
    V_ref = input_transform(x, g)                       # (B, th, tw, M, P1, P1)
    Yh_ref = ewmm(U_ref, V_ref)                         # (B, th, tw, N, P1, P1)
    T = B * g.th * g.tw
    U_std = _to_lib_points(U_ref, n).transpose(2, 1, 0)                     # (P, M, N)
    V_std = _to_lib_points(V_ref.reshape(T, M, g.lv.P1, g.lv.P1), n).transpose(2, 1, 0)
    Yh_std = _to_lib_points(Yh_ref.reshape(T, N, g.lv.P1, g.lv.P1), n).transpose(2, 1, 0)
    U_lib, V_lib, Z_lib = _quads(U_std), _quads(V_std), _level1(Yh_std)

    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        assert plan.info["P"] == U_std.shape[0] and plan.info["T"] == T
        assert plan.info["yhat_bytes"] == 4 * Z_lib.size
        U = torch.empty(plan.u_shape, device="cuda")
        V = torch.full(plan.v_shape, float("nan"), device="cuda")
        Z = torch.full(plan.z_shape, float("nan"), device="cuda")
        y = torch.empty(plan.y_shape, device="cuda")
        plan.kernel_transform(dev(w), U)
        plan.input_transform(dev(x), V)
        torch.cuda.synchronize()
        assert_close(U.cpu().numpy(), U_lib, rel_tol=1e-6, abs_frac=1e-6, what="U")
        # V of the groups no tap reaches is never read, and not written
        live, Vh = live_group_mask(plan.info), V.cpu().numpy()
        lq = np.repeat(live, 4)                         # four quads per group
        assert_close(Vh[lq], V_lib[lq], rel_tol=1e-6, abs_frac=1e-6, what="V")
        assert np.isnan(Vh[~lq]).all()
        # contraction + level-1 output transform, on the oracle's transformed operands
        plan.contract(dev(U_lib), dev(V_lib), Z)
        torch.cuda.synchronize()
        # groups no tap reaches (U zero for every w) are neither computed nor written
        live, Zh = live_group_mask(plan.info), Z.cpu().numpy()
        assert_close(Zh[live], Z_lib[live], rel_tol=1e-5, abs_frac=1e-5, what="Z")
        assert np.isnan(Zh[~live]).all() and not Z_lib[~live].any()
        # output transform levels 2..n alone, on the oracle's Z
        plan.output_transform(dev(Z_lib), y)
        torch.cuda.synchronize()
        assert_close(y.cpu().numpy(), output_transform(Yh_ref, g), rel_tol=1e-6, abs_frac=1e-6,
                     what="y")


# depth 3-4 with N <= 2: the fused kernel.  Tile counts not a multiple of 4
# (a ragged last wavefront), M = 1, 3, 5, 9 (1, 2 and 4 channel groups, some
# of them uneven), padding that reaches past whole windows.
FUSED = [(1, 3, 1, 20, 19, 11, 5), (2, 5, 2, 17, 21, 9, 4), (1, 1, 1, 23, 18, 15, 7),
         (1, 9, 2, 12, 13, 8, 0), (1, 2, 1, 21, 26, 31, 15), (2, 3, 2, 18, 17, 17, 8),
         (1, 5, 1, 33, 16, 16, 0), (2, 4, 1, 70, 45, 9, 4)]


def _stage_refs(case, seed):
    B, M, N, H, W, r, pad = case
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=seed)
    g = geometry(x.shape, w.shape, pad)
    n = g.lv.n
    U_ref = kernel_transform(w, g)
    V_ref = input_transform(x, g)
    Yh_ref = ewmm(U_ref, V_ref)
    T = B * g.th * g.tw
    U_std = _to_lib_points(U_ref, n).transpose(2, 1, 0)
    Yh_std = _to_lib_points(Yh_ref.reshape(T, N, g.lv.P1, g.lv.P1), n).transpose(2, 1, 0)
    return x, w, g, _quads(U_std), _level1(Yh_std), Yh_ref


@pytest.mark.parametrize("case", FUSED, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_fused_input_contract_matches_cpu_nested_reference(case):
    B, M, N, H, W, r, pad = case
    print(f"fused {case}", flush=True)
    x, w, g, U_lib, Z_lib, Yh_ref = _stage_refs(case, seed=11 + r)
    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        assert plan.info["fused_input"] == 1 and plan.info["n"] in (3, 4)
        assert plan.info["workspace_bytes"] == plan.info["u_bytes"] + plan.info["yhat_bytes"]
        Z = torch.full(plan.z_shape, float("nan"), device="cuda")
        plan.input_contract(dev(x), dev(U_lib), Z)
        torch.cuda.synchronize()
        assert_close(Z.cpu().numpy(), Z_lib, rel_tol=1e-5, abs_frac=1e-5, what="Z fused")
        # the unfused stages on the same operands agree
        V = torch.empty(plan.v_shape, device="cuda")
        Z2 = torch.empty(plan.z_shape, device="cuda")
        plan.input_transform(dev(x), V)
        plan.contract(dev(U_lib), V, Z2)
        torch.cuda.synchronize()
        assert_close(Z.cpu().numpy(), Z2.cpu().numpy(), rel_tol=1e-5, abs_frac=1e-5,
                     what="fused vs staged")
        y = torch.empty(plan.y_shape, device="cuda")
        plan.conv2d(dev(x), dev(w), y)
        torch.cuda.synchronize()
        assert_close(y.cpu().numpy(), direct_conv2d(x, w, pad), what=f"y {case}")


def test_fused_input_contract_rejects_other_shapes():
    # buffers of the plan's sizes, so that the library itself refuses the shape
    for shape in [(1, 2, 3, 20, 20, 9, 4),                   # N = 3
                  (1, 2, 1, 20, 20, 7, 3)]:                  # depth 2
        with nwg.Plan(*shape) as plan:
            assert plan.info["fused_input"] == 0
            x = torch.zeros((1, 2, 20, 20), device="cuda")
            U = torch.zeros(plan.u_shape, device="cuda")
            Z = torch.zeros(plan.z_shape, device="cuda")
            with pytest.raises(nwg.NwgError, match="N <= 2"):
                plan.input_contract(x, U, Z)


@pytest.mark.parametrize("N,M,T,depth", [(1, 32, 4096, 1), (5, 5, 100, 1), (128, 128, 256, 1),
                                         (64, 64, 392, 1), (3, 7, 33, 1), (32, 1, 300, 1),
                                         (17, 33, 129, 1), (128, 20, 64, 0), (5, 32, 1000, 0),
                                         (32, 5, 4096, 0), (96, 40, 70, 2),
                                         # full tiles (direct global->LDS path) per tile shape
                                         (64, 32, 128, 1), (16, 16, 128, 2), (32, 48, 256, 1),
                                         (128, 64, 192, 1), (64, 96, 256, 1), (128, 32, 128, 2),
                                         # deep path with a ragged last column tile
                                         (64, 32, 100, 1), (128, 64, 200, 2), (64, 64, 65, 1),
                                         (64, 128, 130, 1), (64, 96, 150, 2), (128, 64, 392, 1),
                                         # persistent deep path (at least 4 tiles per CU slot):
                                         # 64 x 128 tiles, 4 per slot; 64 x 64 tiles with a
                                         # ragged last one and 4 or 5 tiles per slot
                                         (128, 64, 256, 3), (64, 32, 520, 3),
                                         # 128 x 64 blocks (T = 64, N % 128 == 0)
                                         (128, 32, 64, 2), (256, 64, 64, 1)])
def test_contraction_matches_numpy(N, M, T, depth):
    """Z = level-1 A^T of (U[p]^T V[p]) for ragged shapes, through nwg_contract.

    Depth d = 1, 2, 3 (P = 16, 256, 4096) uses B = T images of 2^d x 2^d with
    r = 2^d (one tile each); depth 0 (r = 1) uses one image of 1 x T, where V
    is x and the result is y.
    """
    rng = np.random.default_rng(N * 1000 + M * 10 + T)
    if depth == 0:
        plan = nwg.Plan(1, M, N, 1, T, 1, 0)
        U = rng.standard_normal((M, N))
        V = rng.standard_normal((M, T))
        ref = U.T @ V
        out = torch.empty((N, T), device="cuda")
        plan.contract(dev(U), dev(V), out)
    else:
        side = 2 ** depth
        plan = nwg.Plan(T, M, N, side, side, side, 0)
        P = plan.info["P"]
        assert plan.info["n"] == depth and plan.info["T"] == T
        U = rng.standard_normal((P, M, N))
        V = rng.standard_normal((P, M, T))
        ref = _level1(np.matmul(U.transpose(0, 2, 1), V))
        out = torch.full(plan.z_shape, float("nan"), device="cuda")
        plan.contract(dev(_quads(U)), dev(_quads(V)), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    if depth > 0:
        # the plan computes the groups a tap of its r reaches, whatever U holds
        live = live_group_mask(plan.info)
        assert np.isnan(got[~live]).all()
        got, ref = got[live], ref[live]
    assert_close(got, ref, rel_tol=1e-5, abs_frac=1e-5, what="contract")
    plan.close()


def test_weight_cache_follows_pointer_and_set_weights():
    B, M, N, H, W, r, pad = 1, 3, 4, 14, 14, 5, 2
    _, x, w1 = make_case(B, M, N, H, W, r, pad, seed=1)
    _, _, w2 = make_case(B, M, N, H, W, r, pad, seed=2)
    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        xd = dev(x)
        wd1, wd2 = dev(w1), dev(w2)
        y = torch.empty(plan.y_shape, device="cuda")
        plan.conv2d(xd, wd1, y)
        torch.cuda.synchronize()
        assert_close(y.cpu().numpy(), direct_conv2d(x, w1, pad), what="w1")
        plan.conv2d(xd, wd2, y)                      # new pointer: re-transformed
        torch.cuda.synchronize()
        assert_close(y.cpu().numpy(), direct_conv2d(x, w2, pad), what="w2")
        wd2.copy_(wd1)                                # in place: cache is stale by contract
        plan.set_weights(wd2)
        plan.conv2d(xd, wd2, y)
        torch.cuda.synchronize()
        assert_close(y.cpu().numpy(), direct_conv2d(x, w1, pad), what="set_weights")


def test_depth0_stage_calls_are_rejected():
    with nwg.Plan(1, 2, 2, 8, 8, 1, 0) as plan:
        x = torch.zeros((1, 2, 8, 8), device="cuda")
        with pytest.raises(nwg.NwgError):
            plan.input_transform(x, x)
        with pytest.raises(nwg.NwgError):
            plan.output_transform(x, x)


def test_timing_records_each_stage():
    B, M, N, H, W, r, pad = 1, 8, 8, 32, 32, 7, 3
    _, x, w = make_case(B, M, N, H, W, r, pad, seed=3)
    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        xd, wd = dev(x), dev(w)
        y = torch.empty(plan.y_shape, device="cuda")
        plan.set_timing(True)
        for _ in range(3):
            plan.conv2d(xd, wd, y)
        ms, cnt = plan.get_timing()
        assert cnt == [1, 3, 3, 3]
        assert all(t > 0 for t in ms)
        ms2, cnt2 = plan.get_timing()
        assert cnt2 == [0, 0, 0, 0]


def test_timing_of_the_fused_path_counts_one_launch_as_contraction():
    B, M, N, H, W, r, pad = 1, 4, 1, 32, 32, 9, 4
    _, x, w = make_case(B, M, N, H, W, r, pad, seed=4)
    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        assert plan.info["fused_input"] == 1
        xd, wd = dev(x), dev(w)
        y = torch.empty(plan.y_shape, device="cuda")
        plan.set_timing(True)
        for _ in range(2):
            plan.conv2d(xd, wd, y)
        ms, cnt = plan.get_timing()
        assert cnt == [1, 0, 2, 2]
        assert_close(y.cpu().numpy(), direct_conv2d(x, w, pad), what="fused timing")


def test_two_stream_pipeline_matches_single_stream_bit_for_bit():
    # depth 4, M % 32 == 0, N % 64 == 0, T % 64 == 0: the pipelined path
    B, M, N, H, W, r, pad = 4, 32, 64, 56, 56, 31, 15
    _, x, w = make_case(B, M, N, H, W, r, pad, seed=9, x_dist="normal", w_dist="fanin_normal")
    print("pipeline", flush=True)
    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        assert plan.info["pipeline_parts"] == 1 and plan.info["T"] == 64
        xd, wd = dev(x), dev(w)
        ys = {}
        for parts in (1, 2, 4, 8, 16):
            plan.set_pipeline(parts)
            assert plan.info["pipeline_parts"] == parts
            y = torch.full(plan.y_shape, float("nan"), device="cuda")
            plan.conv2d(xd, wd, y)
            torch.cuda.synchronize()
            ys[parts] = y.cpu().numpy()
        plan.set_timing(True)
        plan.set_pipeline(4)
        plan.conv2d(xd, wd, y)
        ms, cnt = plan.get_timing()
        assert cnt == [0, 4, 4, 1]
        with pytest.raises(nwg.NwgError):
            plan.set_pipeline(3)
    for parts in (2, 4, 8, 16):
        assert np.array_equal(ys[parts], ys[1]), parts
    assert_close(ys[4], direct_conv2d(x, w, pad), what="pipelined y")


def test_pipeline_is_refused_where_it_cannot_split():
    with nwg.Plan(1, 3, 5, 20, 19, 11, 5) as plan:          # depth 3
        assert plan.info["pipeline_parts"] == 1
        with pytest.raises(nwg.NwgError):
            plan.set_pipeline(4)
        plan.set_pipeline(1)


# few channels at depth 1-2: one kernel x -> y (depth 1: M <= 8, N <= 16;
# depth 2: M <= 2, M N <= 64), ragged tiles, B > 1, both paddings
SMALL = [(2, 1, 1, 9, 7, 3, 1), (1, 3, 16, 17, 30, 3, 1), (3, 5, 5, 20, 21, 3, 1),
         (1, 8, 2, 13, 15, 2, 0), (2, 7, 9, 16, 16, 3, 0), (1, 1, 32, 33, 29, 5, 2),
         (2, 2, 7, 18, 19, 7, 3), (1, 1, 64, 16, 16, 4, 0), (2, 2, 32, 21, 22, 6, 0)]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_single_kernel_small_channel_layers(case):
    B, M, N, H, W, r, pad = case
    print(f"small {case}", flush=True)
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=sum(case) + 1)
    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        assert plan.info["fused_conv"] == 1 and plan.info["n"] in (1, 2)
        assert plan.info["workspace_bytes"] == plan.info["u_bytes"]
        plan.set_timing(True)
        y = run_conv(x, w, pad, plan)
        ms, cnt = plan.get_timing()
        assert cnt == [1, 0, 1, 0]
    assert_close(y, direct_conv2d(x, w, pad), what=str(case))


def test_weight_cache_survives_a_freed_weight_tensor():
    """A weight tensor freed after use can hand its memory to the next one:
    the binding keeps the tensor it transformed (and its version counter),
    so a new tensor, or the same one changed in place, is transformed again."""
    B, M, N, H, W, r, pad = 1, 4, 8, 20, 20, 9, 4
    _, x, w1 = make_case(B, M, N, H, W, r, pad, seed=21)
    _, _, w2 = make_case(B, M, N, H, W, r, pad, seed=22)
    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        xd = dev(x)
        y = torch.empty(plan.y_shape, device="cuda")
        plan.conv2d(xd, dev(w1), y)                  # the weight tensor is a temporary
        torch.cuda.synchronize()
        assert_close(y.cpu().numpy(), direct_conv2d(x, w1, pad), what="w1")
        wd2 = dev(w2)                                # may take the freed block's address
        plan.conv2d(xd, wd2, y)
        torch.cuda.synchronize()
        assert_close(y.cpu().numpy(), direct_conv2d(x, w2, pad), what="w2 after w1 freed")
        wd2.copy_(dev(w1))                           # in place, no set_weights
        plan.conv2d(xd, wd2, y)
        torch.cuda.synchronize()
        assert_close(y.cpu().numpy(), direct_conv2d(x, w1, pad), what="w2 changed in place")


def test_allocation_failure_reports_enomem():
    """A plan whose workspace cannot fit on the device (V alone about 2.2 TB
    here) fails with NWG_ENOMEM, releases what it took, and the next plan
    works."""
    lib = nwg.load_library()
    g = nwg.plan_geometry(4096, 128, 128, 56, 56, 31, 15, nwg.NWG_TILE_F2X2_3X3)
    assert g["workspace_bytes"] > 1e12
    free0, _ = torch.cuda.mem_get_info()
    with pytest.raises(nwg.NwgError, match="hipMalloc"):
        nwg.Plan(4096, 128, 128, 56, 56, 31, 15, tile=nwg.NWG_TILE_F2X2_3X3)
    assert lib.nwg_last_status() == nwg.NWG_ENOMEM
    free1, _ = torch.cuda.mem_get_info()
    assert free1 >= free0 - (64 << 20)               # U (4.3 GB) was released
    _, x, w = make_case(1, 2, 3, 12, 12, 5, 2, seed=4)
    with nwg.Plan(1, 2, 3, 12, 12, 5, 2) as plan:
        assert_close(run_conv(x, w, 2, plan), direct_conv2d(x, w, 2), what="after ENOMEM")


def test_bad_device_buffers_are_refused_before_the_library():
    with nwg.Plan(1, 2, 3, 12, 12, 5, 2) as plan:
        x = torch.zeros((1, 2, 12, 12), device="cuda")
        w = torch.zeros((3, 2, 5, 5), device="cuda")
        y = torch.zeros(plan.y_shape, device="cuda")
        with pytest.raises(nwg.NwgError, match="float32"):
            plan.conv2d(x.double(), w, y)
        with pytest.raises(nwg.NwgError, match="contiguous"):
            plan.conv2d(x, w, y.transpose(2, 3))
        with pytest.raises(nwg.NwgError, match="elements"):
            plan.conv2d(x, w, y.reshape(-1)[:-1])
        with pytest.raises(nwg.NwgError, match="aligned"):
            plan.conv2d(torch.zeros(x.numel() + 1, device="cuda")[1:], w, y)
        U = torch.zeros(plan.u_shape, device="cuda")
        with pytest.raises(nwg.NwgError, match="elements"):
            plan.kernel_transform(w, U.reshape(-1)[:-4])


def test_calls_on_a_created_stream_and_the_null_stream():
    """The device check accepts the plan's own device, through a created
    stream and through the NULL stream (the current device's)."""
    B, M, N, H, W, r, pad = 1, 3, 5, 22, 18, 7, 3
    _, x, w = make_case(B, M, N, H, W, r, pad, seed=31)
    ref = direct_conv2d(x, w, pad)
    side = torch.cuda.Stream()
    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        xd, wd = dev(x), dev(w)
        torch.cuda.synchronize()
        for stream in (side, 0):
            y = torch.full(plan.y_shape, float("nan"), device="cuda")
            torch.cuda.synchronize()
            plan.conv2d(xd, wd, y, stream=stream)
            torch.cuda.synchronize()
            assert_close(y.cpu().numpy(), ref, what=f"stream {stream}")
