"""GPU parity of the F(3x3, 3x3) tile (depth 1-2, r <= 9) against the CPU
oracle.

End to end against the fp64 direct convolution (rel-L2 <= 1e-4, max-abs <=
1e-3 max|y|); stage by stage against the oracle's nested transforms on the
same base (Toom-Cook points 0, 1, -1, 2, infinity), re-ordered to the
library's base-5 point order.  Inputs are seeded and synthetic.
"""
import numpy as np
import pytest
import torch

from oracle.direct import direct_conv2d
from oracle.nested import ewmm, geometry, input_transform, kernel_transform, output_transform
from paper_2102_13272_amd import nwg
from paper_2102_13272_amd.workloads import make_case
from tests.gpu_util import assert_close, dev
from tests.layout import f33_base, level1_f33, to_lib_points

pytestmark = pytest.mark.gpu
F33 = nwg.NWG_TILE_F3X3_3X3


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nwg.load_library()          # raises if the HIP library is missing: no fallback


def _conv(x, w, pad):
    B, M, H, W = x.shape
    N, _, r, _ = w.shape
    with nwg.Plan(B, M, N, H, W, r, pad, tile=F33) as plan:
        i = plan.info
        assert i["tile"] == F33 and i["fused_conv"] == 0
        # one output channel at depth 2: the fused kernel, no V; else one or
        # two input channels: the output transform forms the contraction, no Z
        assert i["fused_input"] == (1 if (i["n"] == 2 and N == 1) else 0)
        fo = 1 if (i["n"] >= 1 and M <= 2 and not i["fused_input"]) else 0
        assert i["fused_output"] == fo
        if fo:
            assert i["workspace_bytes"] == i["u_bytes"] + i["v_bytes"]
        y = torch.full(plan.y_shape, float("nan"), device="cuda")
        plan.conv2d(dev(x), dev(w), y)
        torch.cuda.synchronize()
        return y.cpu().numpy().astype(np.float64)


# B, M, N, H, W, r, pad: depth 0-2, ragged tiles and channel blocks (M not a
# multiple of 16, N and T over 64), B > 1, padding past whole windows
E2E = [
    (2, 3, 5, 9, 7, 1, 0),
    (1, 4, 4, 16, 16, 2, 0),
    (2, 5, 3, 11, 13, 3, 1),
    (1, 7, 70, 23, 21, 3, 1),
    (1, 1, 7, 23, 21, 4, 2),
    (3, 6, 4, 17, 30, 5, 2),
    (1, 19, 66, 40, 33, 6, 3),
    (2, 33, 9, 29, 26, 7, 3),
    (1, 3, 2, 15, 15, 8, 0),
    (1, 2, 3, 40, 35, 9, 4),
    (1, 17, 20, 9, 9, 9, 0),      # a single output pixel
    (2, 64, 64, 37, 41, 9, 4),
    # N and T multiples of 4 (the 16-byte loader): M = 64, 32 (whole ring
    # turns per point) and 20 (ragged), several tile blocks, depth 1 and 2
    (4, 64, 68, 26, 26, 7, 3),
    (4, 32, 8, 20, 20, 5, 2),
    (4, 20, 12, 17, 17, 4, 1),
    (4, 64, 64, 30, 30, 3, 1),
    (4, 96, 132, 46, 46, 9, 4),
    # N = 1 at depth 2: the fused kernel (one or several input-channel
    # groups, ragged boxes, M = 1 and odd M)
    (1, 1, 1, 23, 21, 4, 2),
    (2, 5, 1, 40, 35, 9, 4),
    (3, 32, 1, 70, 50, 7, 3),
    (1, 33, 1, 100, 90, 9, 0),
    # one or two input channels: the contraction inside the output transform
    (1, 1, 64, 70, 66, 9, 4),
    (2, 2, 33, 31, 29, 3, 1),
    (1, 2, 5, 44, 40, 7, 3),
]


@pytest.mark.parametrize("case", E2E, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_f33_conv2d_matches_direct_oracle(case):
    B, M, N, H, W, r, pad = case
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=3 * sum(case))
    print(f"f33 case {case}", flush=True)
    assert_close(_conv(x, w, pad), direct_conv2d(x, w, pad), what=str(case))


STAGES = [(1, 3, 4, 12, 10, 3, 1), (2, 4, 3, 13, 11, 6, 2), (1, 5, 2, 20, 19, 9, 4),
          (2, 17, 65, 21, 19, 2, 0), (4, 32, 16, 20, 20, 5, 2), (4, 64, 8, 12, 12, 3, 1)]


@pytest.mark.parametrize("case", STAGES, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_f33_stages_match_cpu_nested_reference(case):
    B, M, N, H, W, r, pad = case
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=5 + r)
    print(f"f33 stages {case}", flush=True)
    g = geometry(x.shape, w.shape, pad, base=f33_base())
    n, P1 = g.lv.n, g.lv.P1
    U_ref = kernel_transform(w, g)                      # (N, M, P1, P1)
    V_ref = input_transform(x, g)                       # (B, th, tw, M, P1, P1)
    Yh_ref = ewmm(U_ref, V_ref)                         # (B, th, tw, N, P1, P1)
    T = B * g.th * g.tw
    U_lib = np.ascontiguousarray(to_lib_points(U_ref, n, 5).transpose(2, 1, 0))   # (P, M, N)
    V_lib = np.ascontiguousarray(
        to_lib_points(V_ref.reshape(T, M, P1, P1), n, 5).transpose(2, 1, 0))       # (P, M, T)
    Yh_lib = to_lib_points(Yh_ref.reshape(T, N, P1, P1), n, 5).transpose(2, 1, 0)  # (P, N, T)
    Z_lib = level1_f33(Yh_lib)

    with nwg.Plan(B, M, N, H, W, r, pad, tile=F33) as plan:
        i = plan.info
        assert (i["n"], i["P"], i["T"], i["Mn"]) == (n, U_lib.shape[0], T, g.lv.Mn)
        assert i["yhat_bytes"] == 4 * Z_lib.size and i["v_bytes"] == 4 * V_lib.size
        U = torch.full(plan.u_shape, float("nan"), device="cuda")
        V = torch.full(plan.v_shape, float("nan"), device="cuda")
        Z = torch.full(plan.z_shape, float("nan"), device="cuda")
        y = torch.full(plan.y_shape, float("nan"), device="cuda")
        plan.kernel_transform(dev(w), U)
        plan.input_transform(dev(x), V)
        torch.cuda.synchronize()
        assert_close(U.cpu().numpy(), U_lib, rel_tol=1e-6, abs_frac=1e-6, what="U")
        assert_close(V.cpu().numpy(), V_lib, rel_tol=1e-6, abs_frac=1e-6, what="V")
        plan.contract(dev(U_lib), dev(V_lib), Z)
        torch.cuda.synchronize()
        assert_close(Z.cpu().numpy(), Z_lib, rel_tol=1e-5, abs_frac=1e-5, what="Z")
        plan.output_transform(dev(Z_lib), y)
        torch.cuda.synchronize()
        # fp32 sums over A^T entries up to 4 on each of four axes (level-1
        # rows, level-2 rows and columns): rounding reaches ~1e-6 of max|y|
        assert_close(y.cpu().numpy(), output_transform(Yh_ref, g), rel_tol=1e-6,
                     abs_frac=1e-5, what="y")


def test_f33_fused_plan_holds_no_v():
    with nwg.Plan(4, 32, 1, 256, 256, 9, 4, tile=F33) as plan:
        i = plan.info
        assert i["fused_input"] == 1 and i["n"] == 2
        z9 = (i["P"] // 25) * 9 * i["T"] * 4
        parts = (i["workspace_bytes"] - i["u_bytes"]) // z9
        assert parts >= 1 and i["workspace_bytes"] == i["u_bytes"] + parts * z9
        assert i["workspace_bytes"] < i["v_bytes"]


def test_f33_rejects_deep_kernels_and_fused_calls():
    with pytest.raises(nwg.NwgError):
        nwg.Plan(1, 2, 2, 20, 20, 10, 0, tile=F33)
    with pytest.raises(nwg.NwgError):
        nwg.Plan(1, 2, 2, 20, 20, 5, 0, tile=F33, depthwise=True)
    with nwg.Plan(1, 3, 1, 30, 30, 9, 4, tile=F33) as plan:
        U = torch.empty(plan.u_shape, device="cuda")
        Z = torch.empty(plan.z_shape, device="cuda")
        x = torch.zeros((1, 3, 30, 30), device="cuda")
        with pytest.raises(nwg.NwgError):
            plan.input_contract(x, U, Z)
        with pytest.raises(nwg.NwgError):
            plan.set_pipeline(2)
