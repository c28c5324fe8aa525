"""nwg_conv2d captured in a HIP graph: every replay equals the eager result.

The library's conv2d path queues kernels only (no allocation, memset or
synchronisation once the weights are transformed), so a caller may capture
it.  The graph is replayed several times, with eager work of the program
and synchronisations between the replays, and each replay is compared with
the eager output bit for bit.  Covers a chain of layers that takes every
kind of launch (fused small-channel kernels, 1x1 GEMMs, the fused F(3,3)
kernel with its partial sums, the three-kernel path, the mixed nest with its
scratch buffer).
"""
import numpy as np
import pytest
import torch

from paper_2102_13272_amd import nwg
from paper_2102_13272_amd.workloads import make_case
from tests.gpu_util import dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nwg.load_library()


# (M, N, r, pad, tile): one chain on 2 x 1 x 64 x 64 inputs
CHAIN = [(1, 32, 5, 2, nwg.NWG_TILE_F2X2_3X3),     # single-kernel depth 2
         (32, 5, 1, 0, nwg.NWG_TILE_F2X2_3X3),     # 1x1 GEMM
         (5, 5, 3, 1, nwg.NWG_TILE_F2X2_3X3),      # single-kernel depth 1
         (5, 64, 7, 3, nwg.NWG_TILE_F2X2_3X3),     # three kernels, depth 2
         (64, 64, 17, 8, nwg.NWG_TILE_MIX_F23_F33),  # mixed nest, depth 4 (scratch)
         (64, 64, 13, 6, nwg.NWG_TILE_MIX_F23_F33),  # mixed nest, depth 3
         (64, 64, 9, 4, nwg.NWG_TILE_F3X3_3X3),    # F(3,3) three kernels
         (64, 1, 9, 4, nwg.NWG_TILE_AUTO)]         # fused F(3,3), partial sums


def test_graph_replays_match_eager():
    B, H, W = 2, 64, 64
    plans, ws, ys = [], [], []
    for i, (M, N, r, pad, tile) in enumerate(CHAIN):
        _, _, w = make_case(B, M, N, H, W, r, pad, seed=100 + i)
        plans.append(nwg.Plan(B, M, N, H, W, r, pad, tile=tile))
        ws.append(dev(w))
        ys.append(torch.empty(plans[-1].y_shape, device="cuda"))
    assert plans[-1].info["tile"] == nwg.NWG_TILE_F3X3_3X3 and plans[-1].info["fused_input"] == 1
    _, x, _ = make_case(B, 1, 1, H, W, 1, 0, seed=7)
    xd = dev(x)

    def step():
        cur = xd
        for p, w, y in zip(plans, ws, ys):
            p.conv2d(cur, w, y)
            cur = y

    step()                                   # transforms the weights (not capturable)
    torch.cuda.synchronize()
    eager = [y.clone() for y in ys]
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=cap):
        step()
    for k in range(4):
        for y in ys:
            y.fill_(float("nan"))            # eager work between the replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(ys, eager)):
            assert torch.equal(a, b), f"replay {k}, layer {i}"
    for p in plans:
        p.close()
