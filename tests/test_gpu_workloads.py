"""GPU parity on the five workloads at full size, in the launch configuration
the benchmark times (one plan per layer, nwg_conv2d on torch's stream).

Every workload is compared with the full fp64 direct oracle, output by
output: the 31x31 workload too, on each path that serves it.
"""
import numpy as np
import pytest
import torch

from oracle.direct import direct_conv2d
from paper_2102_13272_amd import nwg
from paper_2102_13272_amd.workloads import WORKLOADS, make_workload
from tests.gpu_util import assert_close, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nwg.load_library()


def _gpu_layer(plan, x_dev, w):
    y = torch.empty(plan.y_shape, device="cuda")
    plan.conv2d(x_dev, dev(w), y)
    return y


@pytest.mark.parametrize("name", ["c1_r4_valid", "c2_r7", "c3_r13"])
def test_single_layer_workload_full_oracle(name):
    wl = WORKLOADS[name]
    L = wl.layers[0]
    x, (w,) = make_workload(name)
    print(f"workload {name}", flush=True)
    with nwg.Plan(L.B, L.M, L.N, L.H, L.W, L.r, L.pad) as plan:
        y = _gpu_layer(plan, dev(x), w)
        torch.cuda.synchronize()
        assert_close(y.cpu().numpy(), direct_conv2d(x, w, L.pad), what=name)


@pytest.mark.parametrize("name,tile", [("c4_sr_stack", nwg.NWG_TILE_F2X2_3X3),
                                       ("c4_sr_stack", nwg.NWG_TILE_AUTO),
                                       ("srcnn_955", nwg.NWG_TILE_F2X2_3X3),
                                       ("srcnn_955", nwg.NWG_TILE_AUTO),
                                       ("srcnn_955", nwg.NWG_TILE_LD_F2X2_3X3)],
                         ids=["c4_f23", "c4_auto", "srcnn_f23", "srcnn_auto", "srcnn_ld"])
def test_sr_stack_per_layer_and_end_to_end(name, tile):
    wl = WORKLOADS[name]
    x, ws = make_workload(name)
    print(f"workload {name} tile {tile}", flush=True)
    plans = [nwg.Plan(L.B, L.M, L.N, L.H, L.W, L.r, L.pad, tile=tile) for L in wl.layers]
    cur_dev = dev(x)
    ref64 = x.astype(np.float64)
    for i, (L, w, plan) in enumerate(zip(wl.layers, ws, plans)):
        inp = cur_dev.cpu().numpy()
        cur_dev = _gpu_layer(plan, cur_dev, w)
        torch.cuda.synchronize()
        got = cur_dev.cpu().numpy()
        # per layer, on the same fp32 input the GPU saw
        assert_close(got, direct_conv2d(inp, w, L.pad), what=f"layer {i + 1} (r={L.r})")
        ref64 = direct_conv2d(ref64, w, L.pad)
    # end to end against an fp64 chain from the original input
    assert_close(cur_dev.cpu().numpy(), ref64, what="stack end to end")
    for p in plans:
        p.close()


@pytest.mark.parametrize("tile,precision", [(nwg.NWG_TILE_AUTO, nwg.NWG_PRECISION_FP32),
                                            (nwg.NWG_TILE_F2X2_3X3, nwg.NWG_PRECISION_FP32),
                                            (nwg.NWG_TILE_F2X2_3X3, nwg.NWG_PRECISION_BF16_SPLIT)],
                         ids=["auto_mixed_nest", "f23_fp32", "f23_bf16_split"])
def test_large_kernel_workload_whole_output(c5_oracle, tile, precision):
    """Every one of the 6.4 M outputs of the 31x31 workload against the fp64
    direct oracle, on the three paths that serve it: the automatic tile (the
    mixed nest the benchmark times), four F(2,3) levels, and four F(2,3)
    levels with the bf16-split contraction."""
    L, x, w, ref = c5_oracle
    print(f"workload c5_r31 tile {tile} precision {precision}", flush=True)
    with nwg.Plan(L.B, L.M, L.N, L.H, L.W, L.r, L.pad, tile=tile) as plan:
        want_tile = nwg.NWG_TILE_MIX_F23_F33 if tile == nwg.NWG_TILE_AUTO else tile
        assert plan.info["tile"] == want_tile and plan.info["n"] == 4
        plan.set_precision(precision)
        y = torch.full(plan.y_shape, float("nan"), device="cuda")
        plan.conv2d(dev(x), dev(w), y)
        torch.cuda.synchronize()
        got = y.cpu().numpy()
    assert np.isfinite(got).all()
    rel, mabs = assert_close(got, ref, what="c5_r31")
    per_image = [assert_close(got[b], ref[b], what=f"image {b}")[0] for b in range(L.B)]
    print(f"c5_r31 tile {want_tile} precision {precision}: rel-L2 {rel:.3e}, max-abs "
          f"{mabs / np.abs(ref).max():.3e} of max|y|, worst image rel-L2 {max(per_image):.3e}",
          flush=True)
