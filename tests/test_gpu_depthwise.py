"""GPU parity of the depthwise path (Table I's depth-wise row) against the
CPU oracle: end to end against the fp64 direct depthwise correlation, and
stage by stage against the CPU nested reference (kernel transform of
w [C][1][r][r], input transform, element-wise product with the level-1
output transform, fused input+product kernel, output transform).
"""
import numpy as np
import pytest
import torch

from oracle.direct import direct_depthwise_conv2d
from oracle.nested import (depthwise_geometries, ewmm_depthwise, input_transform,
                           kernel_transform, output_transform)
from paper_2102_13272_amd import nwg
from paper_2102_13272_amd.workloads import WORKLOADS, make_case, make_workload
from tests.gpu_util import assert_close, dev
from tests.layout import level1, quads, to_lib_points

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nwg.load_library()


def _run(x, w, pad, plan=None):
    B, C, H, W = x.shape
    r = w.shape[2]
    own = plan is None
    if own:
        plan = nwg.Plan(B, C, C, H, W, r, pad, depthwise=True)
    y = torch.empty(plan.y_shape, device="cuda")
    plan.conv2d(dev(x), dev(w), y)
    torch.cuda.synchronize()
    out = y.cpu().numpy().astype(np.float64)
    if own:
        plan.close()
    return out


# B, C, H, W, r, pad: depths 0..4, ragged tiles, B > 1, valid and same padding
E2E = [(2, 3, 9, 7, 1, 0), (1, 5, 11, 13, 2, 0), (2, 4, 19, 17, 3, 1), (1, 6, 23, 21, 5, 2),
       (3, 5, 17, 30, 7, 3), (1, 7, 21, 18, 9, 4), (2, 3, 29, 26, 13, 6), (1, 4, 40, 35, 31, 15),
       (1, 3, 24, 24, 16, 0), (2, 2, 8, 8, 4, 0)]


@pytest.mark.parametrize("case", E2E, ids=lambda c: "B%d_C%d_%dx%d_r%d_p%d" % c)
def test_depthwise_conv2d_matches_direct_oracle(case):
    B, C, H, W, r, pad = case
    print(f"depthwise {case}", flush=True)
    _, x, w = make_case(B, C, C, H, W, r, pad, seed=sum(case), depthwise=True)
    assert_close(_run(x, w, pad), direct_depthwise_conv2d(x, w, pad), what=str(case))


STAGES = [(2, 3, 14, 13, 5, 2), (1, 4, 20, 19, 11, 5), (1, 2, 24, 20, 31, 15),
          (2, 3, 9, 10, 3, 1)]


@pytest.mark.parametrize("case", STAGES, ids=lambda c: "B%d_C%d_%dx%d_r%d_p%d" % c)
def test_depthwise_stages_match_cpu_nested_reference(case):
    B, C, H, W, r, pad = case
    print(f"depthwise stages {case}", flush=True)
    _, x, w = make_case(B, C, C, H, W, r, pad, seed=5 + r, depthwise=True)
    gk, gx = depthwise_geometries(x.shape, w.shape, pad)
    n = gx.lv.n
    T = B * gx.th * gx.tw
    U_ref = kernel_transform(w, gk)                      # (C, 1, P1, P1)
    V_ref = input_transform(x, gx)                       # (B, th, tw, C, P1, P1)
    Yh_ref = ewmm_depthwise(U_ref, V_ref)
    P1 = gx.lv.P1
    U_lib = quads(to_lib_points(U_ref, n).transpose(2, 1, 0))            # (P/4, 1, C, 4)
    V_lib = quads(to_lib_points(V_ref.reshape(T, C, P1, P1), n).transpose(2, 1, 0))
    Z_lib = level1(to_lib_points(Yh_ref.reshape(T, C, P1, P1), n).transpose(2, 1, 0))
    with nwg.Plan(B, C, C, H, W, r, pad, depthwise=True) as plan:
        assert plan.info["depthwise"] == 1 and plan.info["T"] == T
        assert plan.u_shape == U_lib.shape
        U = torch.empty(plan.u_shape, device="cuda")
        V = torch.empty(plan.v_shape, device="cuda")
        Z = torch.full(plan.z_shape, float("nan"), device="cuda")
        y = torch.empty(plan.y_shape, device="cuda")
        plan.kernel_transform(dev(w), U)
        plan.input_transform(dev(x), V)
        torch.cuda.synchronize()
        assert_close(U.cpu().numpy(), U_lib, rel_tol=1e-6, abs_frac=1e-6, what="U")
        assert_close(V.cpu().numpy(), V_lib, rel_tol=1e-6, abs_frac=1e-6, what="V")
        plan.contract(dev(U_lib), dev(V_lib), Z)
        torch.cuda.synchronize()
        assert_close(Z.cpu().numpy(), Z_lib, rel_tol=1e-5, abs_frac=1e-5, what="Z")
        if n >= 3:
            assert plan.info["fused_input"] == 1
            Z.fill_(float("nan"))
            plan.input_contract(dev(x), dev(U_lib), Z)
            torch.cuda.synchronize()
            assert_close(Z.cpu().numpy(), Z_lib, rel_tol=1e-5, abs_frac=1e-5, what="Z fused")
        plan.output_transform(dev(Z_lib), y)
        torch.cuda.synchronize()
        assert_close(y.cpu().numpy(), output_transform(Yh_ref, gx), rel_tol=1e-6,
                     abs_frac=1e-6, what="y")


def test_depthwise_workload_full_size():
    wl = WORKLOADS["dw7_pnasnet"]
    L = wl.layers[0]
    x, ws = make_workload("dw7_pnasnet")
    print(f"depthwise workload {L}", flush=True)
    with nwg.Plan(L.B, L.M, L.N, L.H, L.W, L.r, L.pad, depthwise=True) as plan:
        y = _run(x, ws[0], L.pad, plan)
    assert_close(y, direct_depthwise_conv2d(x, ws[0], L.pad), what="dw7_pnasnet")


def test_depthwise_rejects_bad_plans():
    with pytest.raises(nwg.NwgError):
        nwg.Plan(1, 3, 3, 8, 8, 1, 1, depthwise=True)      # r = 1 with padding
    with pytest.raises(ValueError):
        nwg.Plan(1, 3, 4, 8, 8, 3, 1, depthwise=True)      # M != N
