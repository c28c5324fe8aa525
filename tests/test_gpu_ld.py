"""GPU parity of the linear-decomposition plans (NWG_TILE_LD_F2X2_3X3).

Sec. II.B: the r x r kernel is cut into ceil(r/3)^2 sub-kernels of 3 x 3,
each meets the input window moved by its offset, and the Winograd-domain
products are summed before one output transform.  Exact in exact
arithmetic, so the library's fp32 result is held to the same bar as the
nested path against the fp64 direct oracle; on small shapes the oracle's own
linear-decomposition loop agrees with the direct oracle, which ties the
GPU path to Sec. II.B's construction as well.  The transformed sub-kernels
are checked against G w_sub G^T.
"""
import numpy as np
import pytest
import torch

from oracle.direct import direct_conv2d
from oracle.lindecomp import ld_conv2d
from oracle.nested import base_f23
from paper_2102_13272_amd import nwg
from paper_2102_13272_amd.workloads import make_case
from tests.gpu_util import assert_close, dev

pytestmark = pytest.mark.gpu
LD = nwg.NWG_TILE_LD_F2X2_3X3


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nwg.load_library()


# B, M, N, H, W, r, pad: c = 1..11 sub-kernels per axis, ragged tiles and
# channel blocks, deep-path contraction shapes (M c^2 % 32 == 0, N % 64 == 0)
E2E = [
    (1, 3, 5, 11, 9, 2, 0),
    (2, 4, 3, 13, 12, 4, 1),
    (1, 5, 7, 20, 19, 7, 3),
    (2, 2, 3, 17, 23, 9, 4),
    (1, 3, 2, 30, 27, 13, 6),
    (1, 2, 4, 40, 36, 31, 15),
    (2, 8, 64, 24, 24, 6, 2),        # M c^2 = 32: deep contraction
    (1, 32, 64, 28, 28, 9, 4),       # M c^2 = 288
]


@pytest.mark.parametrize("case", E2E, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_ld_conv2d_matches_direct_oracle(case):
    B, M, N, H, W, r, pad = case
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=31 * sum(case))
    print(f"ld case {case}", flush=True)
    with nwg.Plan(B, M, N, H, W, r, pad, tile=LD) as plan:
        assert plan.info["ld_c"] == -(-r // 3) and plan.info["n"] == 1
        y = torch.full(plan.y_shape, float("nan"), device="cuda")
        plan.conv2d(dev(x), dev(w), y)
        torch.cuda.synchronize()
        got = y.cpu().numpy().astype(np.float64)
    assert_close(got, direct_conv2d(x, w, pad), what=str(case))


def test_ld_oracle_loop_agrees_on_a_small_case():
    B, M, N, H, W, r, pad = 1, 2, 2, 10, 9, 7, 3
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=5)
    ref_ld = ld_conv2d(x, w, pad)
    np.testing.assert_allclose(ref_ld, direct_conv2d(x, w, pad), rtol=1e-10, atol=1e-10)
    with nwg.Plan(B, M, N, H, W, r, pad, tile=LD) as plan:
        y = torch.empty(plan.y_shape, device="cuda")
        plan.conv2d(dev(x), dev(w), y)
        torch.cuda.synchronize()
        assert_close(y.cpu().numpy().astype(np.float64), ref_ld, what="vs LD loop")


def test_ld_kernel_transform_is_g_wsub_gt():
    B, M, N, H, W, r, pad = 1, 3, 4, 20, 20, 8, 0          # c = 3: sub-kernels padded
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=9)
    G = base_f23().G.astype(np.float64)
    c = 3
    wp = np.zeros((N, M, 3 * c, 3 * c))
    wp[:, :, :r, :r] = w
    with nwg.Plan(B, M, N, H, W, r, pad, tile=LD) as plan:
        U = torch.empty(plan.u_shape, device="cuda")
        plan.kernel_transform(dev(w), U)
        torch.cuda.synchronize()
        Ul = U.cpu().numpy().astype(np.float64)             # [4][M c^2][N][4]
    for cu in range(c):
        for cv in range(c):
            sub = wp[:, :, 3 * cu:3 * cu + 3, 3 * cv:3 * cv + 3]
            ref = np.einsum("pa,nmab,qb->pqmn", G, sub, G)  # [q1r][q1c][m][n]
            mv = (cu * c + cv) * M + np.arange(M)
            got = Ul[:, mv, :, :].transpose(0, 3, 1, 2)    # [q1r][q1c][m][n]
            assert_close(got, ref, rel_tol=1e-6, abs_frac=1e-6, what=f"U sub ({cu},{cv})")


def test_ld_is_rejected_for_depthwise_and_split():
    with pytest.raises(nwg.NwgError):
        nwg.Plan(1, 4, 4, 20, 20, 7, 3, tile=LD, depthwise=True)
    with nwg.Plan(1, 32, 64, 40, 40, 7, 3, tile=LD) as plan:
        with pytest.raises(nwg.NwgError):
            plan.set_precision(nwg.NWG_PRECISION_BF16_SPLIT)
        x = torch.zeros((1, 32, 40, 40), device="cuda")
        U = torch.zeros(plan.u_shape, device="cuda")
        Z = torch.zeros(plan.z_shape, device="cuda")
        with pytest.raises(nwg.NwgError, match="N <= 2"):
            plan.input_contract(x, U, Z)
