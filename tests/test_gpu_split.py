"""GPU parity of the bf16-split contraction (NWG_PRECISION_BF16_SPLIT).

Every U and V value is carried as hi + lo, two bf16 halves of one word; the
contraction takes all four partial products on bf16 MFMA with fp32
accumulation.  The tests compare against the fp64 oracle: the split stages
(the input transform's pairs against the oracle's V; the contraction against
the oracle's Winograd-domain product), and whole convolutions at depths 1-4
against the direct oracle with the same bar as the fp32 path (rel-L2 <= 1e-4,
max-abs <= 1e-3 max|y|).  The host-side split below is test infrastructure:
numpy bit arithmetic following the format's definition (round to nearest
even on the upper 16 bits of an fp32 word).
"""
import numpy as np
import pytest
import torch

from oracle.direct import direct_conv2d
from oracle.nested import ewmm, geometry, input_transform, kernel_transform
from paper_2102_13272_amd import nwg
from paper_2102_13272_amd.workloads import make_case
from tests.gpu_util import assert_close, dev, errors
from tests.layout import level1 as _level1, quads as _quads, to_lib_points as _to_lib_points

pytestmark = pytest.mark.gpu
SPLIT = nwg.NWG_PRECISION_BF16_SPLIT


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    nwg.load_library()          # raises if the HIP library is missing: no fallback


def _bf16_rne(bits32):
    """uint32 fp32 bit patterns -> the upper 16 bits rounded to nearest even."""
    b = bits32.astype(np.uint64)
    return ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint32) & 0xFFFF


def split_pairs(a):
    """fp32 array -> packed (hi | lo << 16) words, as float32 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    hi = _bf16_rne(a.view(np.uint32))
    rem = (a - (hi << 16).view(np.float32)).astype(np.float32)
    lo = _bf16_rne(rem.view(np.uint32))
    return (hi | (lo << 16)).astype(np.uint32).view(np.float32)


def unsplit(words):
    """packed words (as float32 bit patterns) -> hi + lo in float64."""
    u = np.ascontiguousarray(words).view(np.uint32)
    hi = (u & 0xFFFF) << 16
    lo = (u >> 16) << 16
    return hi.astype(np.uint32).view(np.float32).astype(np.float64) + \
        lo.astype(np.uint32).view(np.float32).astype(np.float64)


def test_host_split_is_the_format():
    # hi is the nearest bf16 (ties to even), lo the nearest bf16 of the rest
    v = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -9, -3.14159265, 1e-20, 0.0],
                 dtype=np.float32)
    w = split_pairs(v).view(np.uint32)
    hi = ((w & 0xFFFF) << 16).view(np.float32)
    assert hi[0] == 1.0 and hi[1] == 1.0                       # tie -> even (1.0)
    assert hi[2] == np.float32(1.0 + 2.0 ** -7)                # 1.0117 rounds up
    assert abs(unsplit(split_pairs(v)) - v.astype(np.float64)).max() <= 2.0 ** -16 * 3.2


# B, M, N, H, W, r, pad: depth 1-4; T a multiple of 128 (64 x 128 tiles) or
# not (64 x 64 tiles with a ragged last one); N = 64, 128; M = 32, 64
E2E = [
    (1, 32, 64, 24, 24, 3, 1),      # depth 1, T = 144
    (2, 64, 64, 16, 16, 2, 0),      # depth 1, T = 128
    (1, 32, 128, 32, 32, 7, 3),     # depth 2, T = 64
    (2, 64, 64, 30, 30, 5, 2),      # depth 2, T = 128
    (1, 32, 64, 64, 64, 9, 4),      # depth 3, T = 64
    (2, 32, 64, 40, 40, 13, 6),     # depth 3, T = 50 -> rejected (T < 64)
    (4, 32, 64, 64, 64, 17, 8),     # depth 4, T = 64
    (4, 64, 64, 48, 48, 31, 15),    # depth 4, T = 36 -> rejected
]


@pytest.mark.parametrize("case", E2E, ids=lambda c: "B%d_M%d_N%d_%dx%d_r%d_p%d" % c)
def test_split_conv2d_matches_direct_oracle(case):
    B, M, N, H, W, r, pad = case
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=sum(case), x_dist="normal",
                        w_dist="fanin_normal")
    print(f"split case {case}", flush=True)
    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        if plan.info["T"] < 64:
            with pytest.raises(nwg.NwgError, match="split precision"):
                plan.set_precision(SPLIT)
            assert plan.info["precision"] == nwg.NWG_PRECISION_FP32
            return
        plan.set_precision(SPLIT)
        assert plan.info["precision"] == SPLIT
        y = torch.full(plan.y_shape, float("nan"), device="cuda")
        plan.conv2d(dev(x), dev(w), y)
        torch.cuda.synchronize()
        got = y.cpu().numpy().astype(np.float64)
    ref = direct_conv2d(x, w, pad)
    rel, mabs, scale = errors(got, ref)
    print(f"  split rel-L2 {rel:.2e}, max-abs {mabs / scale:.2e} of max|y|", flush=True)
    assert_close(got, ref, what=str(case))


def test_split_stages_match_cpu_nested_reference():
    B, M, N, H, W, r, pad = 2, 32, 64, 30, 30, 5, 2      # depth 2, T = 128
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=77)
    g = geometry(x.shape, w.shape, pad)
    n = g.lv.n
    U_ref = kernel_transform(w, g)
    V_ref = input_transform(x, g)
    Yh_ref = ewmm(U_ref, V_ref)
    T = B * g.th * g.tw
    U_std = _to_lib_points(U_ref, n).transpose(2, 1, 0)                        # (P, M, N)
    V_std = _to_lib_points(V_ref.reshape(T, M, g.lv.P1, g.lv.P1), n).transpose(2, 1, 0)
    Yh_std = _to_lib_points(Yh_ref.reshape(T, N, g.lv.P1, g.lv.P1), n).transpose(2, 1, 0)
    U_q, V_q, Z_ref = _quads(U_std), _quads(V_std), _level1(Yh_std)
    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        plan.set_precision(SPLIT)
        U = torch.empty(plan.u_shape, device="cuda")
        V = torch.empty(plan.v_shape, device="cuda")
        Z = torch.full(plan.z_shape, float("nan"), device="cuda")
        plan.kernel_transform(dev(w), U)
        plan.input_transform(dev(x), V)
        torch.cuda.synchronize()
        # the stored pairs carry 16 significant bits of each transformed value
        assert_close(unsplit(U.cpu().numpy()), U_q, rel_tol=2e-5, abs_frac=2e-5, what="U pairs")
        assert_close(unsplit(V.cpu().numpy()), V_q, rel_tol=2e-5, abs_frac=2e-5, what="V pairs")
        # the contraction on the oracle's operands, split on the host
        plan.contract(dev(split_pairs(U_q)), dev(split_pairs(V_q)), Z)
        torch.cuda.synchronize()
        assert_close(Z.cpu().numpy(), Z_ref, rel_tol=5e-5, abs_frac=5e-5, what="Z split")


@pytest.mark.parametrize("ubits,vbits", [(10, 6), (6, 10)])
def test_split_contraction_of_exact_pairs_is_exact(ubits, vbits):
    # integer-valued operands (scaled by powers of two): a 10-bit integer
    # needs both halves (hi + lo), a 6-bit one fits hi alone; every partial
    # product and every fp32 partial sum is then an integer below 2^24, so
    # the split contraction must reproduce the exact result
    B, M, N = 128, 32, 64
    rng = np.random.default_rng(5 + ubits)
    with nwg.Plan(B, M, N, 2, 2, 2, 0) as plan:        # depth 1, T = 128, P = 16
        plan.set_precision(SPLIT)
        P = plan.info["P"]
        U = rng.integers(-(2 ** ubits - 1), 2 ** ubits, (P, M, N)).astype(np.float64) / 64
        V = rng.integers(-(2 ** vbits - 1), 2 ** vbits, (P, M, 128)).astype(np.float64) / 32
        assert np.abs(unsplit(split_pairs(U)) - U).max() == 0.0
        ref = _level1(np.einsum("pmn,pmt->pnt", U, V))
        Z = torch.empty(plan.z_shape, device="cuda")
        plan.contract(dev(split_pairs(_quads(U))), dev(split_pairs(_quads(V))), Z)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(Z.cpu().numpy().astype(np.float64), ref)


def test_precision_switch_invalidates_weights_and_round_trips():
    B, M, N, H, W, r, pad = 2, 32, 64, 30, 30, 5, 2
    L, x, w = make_case(B, M, N, H, W, r, pad, seed=3)
    with nwg.Plan(B, M, N, H, W, r, pad) as plan:
        xd, wd = dev(x), dev(w)
        y0 = torch.empty(plan.y_shape, device="cuda")
        y1 = torch.empty(plan.y_shape, device="cuda")
        y2 = torch.empty(plan.y_shape, device="cuda")
        plan.conv2d(xd, wd, y0)
        plan.set_precision(SPLIT)
        plan.conv2d(xd, wd, y1)            # same w pointer: the weights must be re-split
        plan.set_precision(nwg.NWG_PRECISION_FP32)
        plan.conv2d(xd, wd, y2)
        torch.cuda.synchronize()
        a, b, c = (t.cpu().numpy() for t in (y0, y1, y2))
    np.testing.assert_array_equal(a, c)
    assert not np.array_equal(a, b)
    ref = direct_conv2d(x, w, pad)
    assert_close(b.astype(np.float64), ref, what="split after fp32")


def test_split_precision_rejections():
    with nwg.Plan(1, 16, 64, 40, 40, 5, 2) as plan:       # M % 32 != 0
        with pytest.raises(nwg.NwgError, match="split precision"):
            plan.set_precision(SPLIT)
    with nwg.Plan(1, 32, 32, 40, 40, 5, 2) as plan:       # N % 64 != 0
        with pytest.raises(nwg.NwgError, match="split precision"):
            plan.set_precision(SPLIT)
    with nwg.Plan(1, 32, 2, 64, 64, 9, 4) as plan:        # fused N <= 2
        with pytest.raises(nwg.NwgError):
            plan.set_precision(SPLIT)
    with nwg.Plan(1, 32, 64, 40, 40, 5, 2, tile=nwg.NWG_TILE_F3X3_3X3) as plan:
        with pytest.raises(nwg.NwgError):
            plan.set_precision(SPLIT)
    with nwg.Plan(1, 32, 64, 40, 40, 5, 2) as plan:
        with pytest.raises(nwg.NwgError):
            plan.set_precision(7)
