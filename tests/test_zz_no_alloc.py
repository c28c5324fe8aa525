"""nwg_conv2d_noalloc (the entry point that allocates nothing) against
nwg_conv2d on a plan of the same arguments, through the C ABI: the same
kernels on the same inputs must give the same output, bit for bit, on two
calls in a row (the second smaller, so it runs on what the first left in the
static scratch), and both within the fp32 bar of the fp64 oracle."""
import ctypes

import numpy as np
import pytest
import torch

from oracle.direct import direct_conv2d
from paper_2102_13272_amd import nwg
from paper_2102_13272_amd.workloads import make_case
from tests.gpu_util import assert_close, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nwg.load_library()


def _noalloc(lib, x, w, y, pad, tile):
    B, M, H, W = x.shape
    N, _, r, _ = w.shape
    s = torch.cuda.current_stream().cuda_stream
    return lib.nwg_conv2d_noalloc(B, M, N, H, W, r, pad, tile, x.data_ptr(), w.data_ptr(),
                                  y.data_ptr(), s)


# (B, M, N, H, W, r, pad, tile): the first fills most of the 64 MiB (the 7x7
# 32->32 64x64 workload layer, then the mixed nest at depth 3 with its
# scratch-free Z), the second is smaller and lands on the first's leftovers
SEQUENCES = [
    [(1, 32, 32, 64, 64, 7, 3, nwg.NWG_TILE_F2X2_3X3), (1, 5, 7, 30, 26, 13, 6, nwg.NWG_TILE_F2X2_3X3)],
    [(2, 16, 24, 40, 40, 13, 6, nwg.NWG_TILE_MIX_F23_F33), (1, 3, 2, 22, 19, 5, 2, nwg.NWG_TILE_AUTO)],
    [(1, 64, 64, 32, 32, 9, 4, nwg.NWG_TILE_F3X3_3X3), (2, 8, 16, 17, 23, 1, 0, nwg.NWG_TILE_AUTO)],
    # the fused kernels: x, U -> Z without V (depth 3, N = 2), then the F(3,3)
    # one-output-channel kernel with its partial sums, then one kernel x -> y
    [(1, 8, 2, 40, 40, 11, 5, nwg.NWG_TILE_F2X2_3X3), (1, 3, 1, 30, 30, 9, 4, nwg.NWG_TILE_AUTO),
     (1, 2, 3, 22, 19, 5, 2, nwg.NWG_TILE_AUTO)],
]


@pytest.mark.parametrize("seq", SEQUENCES,
                         ids=["f23", "mixed_then_auto", "f33_then_depth0", "fused_kernels"])
def test_noalloc_matches_conv2d_on_two_calls_in_a_row(seq):
    lib = nwg.load_library()
    for k, (B, M, N, H, W, r, pad, tile) in enumerate(seq):
        print(f"noalloc call {k}: {(B, M, N, H, W, r, pad, tile)}", flush=True)
        _, x, w = make_case(B, M, N, H, W, r, pad, seed=100 + 7 * k + r)
        xd, wd = dev(x), dev(w)
        with nwg.Plan(B, M, N, H, W, r, pad, tile=tile) as plan:
            assert plan.info["workspace_bytes"] <= nwg.NWG_NOALLOC_SCRATCH_BYTES
            y_ref = torch.full(plan.y_shape, float("nan"), device="cuda")
            plan.conv2d(xd, wd, y_ref)
            y = torch.full(plan.y_shape, float("nan"), device="cuda")
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        assert _noalloc(lib, xd, wd, y, pad, tile) == nwg.NWG_OK, nwg.last_error()
        torch.cuda.synchronize()
        # nothing allocated: at most the library's code object with its static
        # array, loaded on the device's first call
        drop = free0 - torch.cuda.mem_get_info()[0]
        assert drop <= (nwg.NWG_NOALLOC_SCRATCH_BYTES + (16 << 20) if k == 0 else 0), drop
        got, ref = y.cpu().numpy(), y_ref.cpu().numpy()
        assert np.isfinite(got).all()
        assert np.array_equal(got, ref), f"call {k}: differs from nwg_conv2d"
        assert_close(got, direct_conv2d(x, w, pad), what=f"call {k}")


def test_noalloc_refuses_what_does_not_fit_and_queues_nothing():
    lib = nwg.load_library()
    B, M, N, H, W, r, pad = 8, 64, 64, 56, 56, 13, 6       # 581 MB of workspace
    x = torch.zeros((B, M, H, W), device="cuda")
    w = torch.zeros((N, M, r, r), device="cuda")
    y = torch.full((B, N, H, W), 7.0, device="cuda")
    rc = _noalloc(lib, x, w, y, pad, nwg.NWG_TILE_F2X2_3X3)
    assert rc == nwg.NWG_EUNSUPPORTED and "static scratch" in nwg.last_error()
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())
    assert lib.nwg_conv2d_noalloc(1, 1, 1, 8, 8, 3, 1, 0, None, None, None, None) == nwg.NWG_EINVAL


def test_noalloc_binding_wrapper():
    B, M, N, H, W, r, pad = 1, 4, 6, 18, 18, 4, 0
    _, x, w = make_case(B, M, N, H, W, r, pad, seed=5)
    y = torch.empty((B, N, H - r + 1, W - r + 1), device="cuda")
    nwg.conv2d_noalloc(dev(x), dev(w), y, pad)
    torch.cuda.synchronize()
    assert_close(y.cpu().numpy(), direct_conv2d(x, w, pad), what="wrapper")
