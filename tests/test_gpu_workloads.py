"""GPU parity on the five workloads at full size, in the launch configuration
the benchmark times (one plan per layer, nwg_conv2d on torch's stream).

Small workloads are compared with the full fp64 direct oracle; the 31x31
workload with a sample of outputs computed one by one, plus checks that hold
at any size (every output finite, the ragged tile edges included).
"""
import numpy as np
import pytest
import torch

from oracle.direct import direct_conv2d, direct_conv2d_points
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


@pytest.mark.parametrize("precision", [nwg.NWG_PRECISION_FP32, nwg.NWG_PRECISION_BF16_SPLIT],
                         ids=["fp32", "bf16_split"])
def test_large_kernel_workload_sampled(precision):
    name = "c5_r31"
    L = WORKLOADS[name].layers[0]
    x, (w,) = make_workload(name)
    print(f"workload {name} precision {precision}", flush=True)
    with nwg.Plan(L.B, L.M, L.N, L.H, L.W, L.r, L.pad) as plan:
        plan.set_precision(precision)
        y = _gpu_layer(plan, dev(x), w)
        torch.cuda.synchronize()
        yh = y.cpu().numpy()
    assert np.isfinite(yh).all()
    rng = np.random.default_rng(5)
    pts = {(int(rng.integers(L.B)), int(rng.integers(L.N)), int(rng.integers(L.Ho)),
            int(rng.integers(L.Wo))) for _ in range(1500)}
    # corners and the last rows/columns of the ragged-free 4x4 tile grid
    for b in (0, L.B - 1):
        for n in (0, L.N - 1):
            for i in (0, 15, 16, L.Ho - 1):
                for j in (0, 15, 16, L.Wo - 1):
                    pts.add((b, n, i, j))
    pts = sorted(pts)
    ref = direct_conv2d_points(x, w, L.pad, pts)
    got = np.array([yh[p] for p in pts], dtype=np.float64)
    assert_close(got, ref, what=name)
