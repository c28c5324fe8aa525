"""Seeded random convolutions through nwg_conv2d against the fp64 direct
oracle, whole outputs: every tile (F(2x2,3x3), F(3x3,3x3), the linear
decomposition, the mixed nest, the automatic choice), dense and depthwise
plans, kernel sizes 1 to 39, padding from none to r - 1, ragged tile grids,
channel counts that are and are not multiples of the kernels' blocks.
Shapes a tile does not serve (nwg_plan_geometry says so) are drawn again.
"""
import numpy as np
import pytest
import torch

from oracle.direct import direct_conv2d, direct_depthwise_conv2d
from paper_2102_13272_amd import nwg
from tests.gpu_util import assert_close, dev

pytestmark = pytest.mark.gpu

TILES = [nwg.NWG_TILE_F2X2_3X3, nwg.NWG_TILE_F3X3_3X3, nwg.NWG_TILE_LD_F2X2_3X3,
         nwg.NWG_TILE_MIX_F23_F33, nwg.NWG_TILE_AUTO]
R_MAX = {nwg.NWG_TILE_F2X2_3X3: 31, nwg.NWG_TILE_F3X3_3X3: 9, nwg.NWG_TILE_LD_F2X2_3X3: 21,
         nwg.NWG_TILE_MIX_F23_F33: 39, nwg.NWG_TILE_AUTO: 31}


def _draw(seed):
    """One servable case: (B, M, N, H, W, r, pad, tile, depthwise)."""
    rng = np.random.default_rng(seed)
    while True:
        tile = TILES[int(rng.integers(len(TILES)))]
        depthwise = bool(rng.random() < 0.4) and tile in (nwg.NWG_TILE_F2X2_3X3,
                                                          nwg.NWG_TILE_AUTO)
        r = int(rng.integers(1, R_MAX[tile] + 1))
        pad = int(rng.integers(0, r)) if r > 1 else 0
        B = int(rng.integers(1, 4))
        M = int(rng.choice([1, 2, 3, 5, 8, 16, 17, 32, 33, 64]))
        N = M if depthwise else int(rng.choice([1, 2, 3, 7, 16, 20, 32, 64]))
        lo = max(1, r - 2 * pad)
        H = int(rng.integers(lo, lo + 60))
        W = int(rng.integers(lo, lo + 60))
        # keep the oracle's work small
        if (B * M * H * W * r * r if depthwise else B * M * N * H * W * r * r) > 4e8:
            continue
        try:
            if depthwise:
                nwg.plan_geometry_depthwise(B, M, H, W, r, pad, tile)
            else:
                nwg.plan_geometry(B, M, N, H, W, r, pad, tile)
        except nwg.NwgError:
            continue
        if r == 1 and pad:
            continue
        return B, M, N, H, W, r, pad, tile, depthwise


CASES = [_draw(s) for s in range(128)]


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nwg.load_library()


@pytest.mark.parametrize("case", CASES,
                         ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d_t%d_dw%d" % (*c[:8], c[8]))
def test_random_convolution_matches_oracle(case):
    B, M, N, H, W, r, pad, tile, depthwise = case
    rng = np.random.default_rng(hash(case) % (1 << 32))
    x = rng.standard_normal((B, M, H, W)).astype(np.float32)
    w = (rng.standard_normal((N, 1 if depthwise else M, r, r)) /
         np.sqrt((1 if depthwise else M) * r * r)).astype(np.float32)
    print(f"fuzz case {case}", flush=True)
    with nwg.Plan(B, M, N, H, W, r, pad, tile=tile, depthwise=depthwise) as plan:
        y = torch.full(plan.y_shape, float("nan"), device="cuda")
        plan.conv2d(dev(x), dev(w), y)
        torch.cuda.synchronize()
        got = y.cpu().numpy()
    ref = (direct_depthwise_conv2d if depthwise else direct_conv2d)(x, w, pad)
    assert_close(got, ref, what=str(case))
