"""CPU checks of the C ABI: the library loads, exports every declared symbol,
and its host-side plan geometry matches the oracle's level recurrence
(two independent implementations of Sec. III.B's nesting).  No device work.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle.nested import base_f23, nesting_levels
from paper_2102_13272_amd import nwg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nwg.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nwg_[a-z_0-9]+)\s*\(", text)))


def test_library_loads_and_exports_every_declared_symbol():
    lib = nwg.load_library()
    declared = _declared_functions()
    assert len(declared) >= 15
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(n for n, _, _ in nwg.SIGNATURES) == declared
    assert lib.nwg_version().decode().startswith("nwg")


def test_info_struct_layout_matches_header():
    # the binding's struct must have the same fields, in order, as the header
    text = open(HEADER).read()
    body = text[text.index("typedef struct nwg_plan_info"):text.index("} nwg_plan_info;")]
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    names = []
    for decl in body.split(";")[:-1]:
        decl = decl.split("{")[-1]
        for part in decl.split(","):
            m = re.search(r"([A-Za-z_][A-Za-z_0-9]*)\s*(\[[^\]]*\])?\s*$", part.strip())
            if m:
                names.append(m.group(1))
    assert names == [f for f, _ in nwg.nwg_plan_info._fields_]


@pytest.mark.parametrize("r", list(range(1, 32)))
def test_geometry_matches_oracle_levels(r):
    B, M, N, H, W = 2, 3, 5, 40, 37
    pad = (r - 1) // 2
    g = nwg.plan_geometry(B, M, N, H, W, r, pad)
    lv = nesting_levels(base_f23(), r)
    assert g["n"] == lv.n and g["Mn"] == lv.Mn and g["Kn"] == lv.Kn
    assert g["strides"] == lv.strides
    if lv.n:
        assert g["Ln"] == lv.Ln
    Ho, Wo = H + 2 * pad - r + 1, W + 2 * pad - r + 1
    assert (g["Ho"], g["Wo"]) == (Ho, Wo)
    th, tw = -(-Ho // lv.Mn), -(-Wo // lv.Mn)
    assert (g["th"], g["tw"], g["T"]) == (th, tw, B * th * tw)
    P = 4 ** (2 * lv.n)
    assert g["P"] == P
    if lv.n:
        assert g["u_bytes"] == 4 * P * M * N
        assert g["v_bytes"] == 4 * P * M * B * th * tw
        assert g["yhat_bytes"] == 4 * (P // 4) * N * B * th * tw     # after the level-1 output step
        assert g["ewmm_mults"] == P * B * th * tw * M * N
    assert g["direct_flop"] == 2 * B * N * M * Ho * Wo * r * r


def test_geometry_of_the_five_workloads():
    from paper_2102_13272_amd.workloads import WORKLOADS
    expect = {"c1_r4_valid": [(2, 16, 256)], "c2_r7": [(2, 256, 256)], "c3_r13": [(3, 392, 4096)],
              "c5_r31": [(4, 256, 65536)],
              "c4_sr_stack": [(2, 16384, 256), (0, 65536, 1)] + [(1, 65536, 16)] * 4
              + [(0, 65536, 1), (3, 4096, 4096)],
              "dw7_pnasnet": [(2, 8 * 21 * 21, 256)],
              "srcnn_955": [(3, 32 * 32, 4096), (2, 64 * 64, 256), (2, 64 * 64, 256)]}
    for name, wl in WORKLOADS.items():
        got = []
        for L in wl.layers:
            if L.depthwise:
                g = nwg.plan_geometry_depthwise(L.B, L.M, L.H, L.W, L.r, L.pad)
            else:
                g = nwg.plan_geometry(L.B, L.M, L.N, L.H, L.W, L.r, L.pad)
            got.append((g["n"], g["T"] if g["n"] else g["Ho"] * g["Wo"], g["P"]))
        assert got == expect[name], name
    g = nwg.plan_geometry(16, 128, 128, 56, 56, 31, 15)
    assert g["workspace_bytes"] == (4 + 8 + 2) * 2 ** 30


@pytest.mark.parametrize("args,rc", [
    ((0, 1, 1, 8, 8, 3, 0, 0), nwg.NWG_EINVAL),       # empty batch
    ((1, 0, 1, 8, 8, 3, 0, 0), nwg.NWG_EINVAL),
    ((1, 1, 0, 8, 8, 3, 0, 0), nwg.NWG_EINVAL),
    ((1, 1, 1, 0, 8, 3, 0, 0), nwg.NWG_EINVAL),
    ((1, 1, 1, 8, 8, 0, 0, 0), nwg.NWG_EINVAL),
    ((1, 1, 1, 8, 8, 3, -1, 0), nwg.NWG_EINVAL),
    ((1, 1, 1, 4, 4, 9, 0, 0), nwg.NWG_EINVAL),       # kernel larger than the input
    ((1, 1, 1, 64, 64, 32, 0, 0), nwg.NWG_EUNSUPPORTED),  # depth 5
    ((1, 1, 1, 8, 8, 3, 1, 7), nwg.NWG_EUNSUPPORTED),    # unknown tile
])
def test_geometry_rejects_bad_arguments(args, rc):
    lib = nwg.load_library()
    info = nwg.nwg_plan_info()
    assert lib.nwg_plan_geometry(*args, ctypes.byref(info)) == rc
    assert lib.nwg_last_error().decode() != ""


def test_null_arguments_are_rejected_without_a_device():
    lib = nwg.load_library()
    assert lib.nwg_plan_query(None, None) == nwg.NWG_EINVAL
    assert lib.nwg_conv2d(None, None, None, None, None) == nwg.NWG_EINVAL
    assert lib.nwg_contract(None, None, None, None, None) == nwg.NWG_EINVAL
    assert lib.nwg_plan_set_timing(None, 1) == nwg.NWG_EINVAL
    lib.nwg_plan_destroy(None)                       # NULL-safe
    # a NULL geometry output on every tile, the automatic choice included
    for tile in (nwg.NWG_TILE_F2X2_3X3, nwg.NWG_TILE_F3X3_3X3, nwg.NWG_TILE_LD_F2X2_3X3,
                 nwg.NWG_TILE_MIX_F23_F33, nwg.NWG_TILE_AUTO):
        assert lib.nwg_plan_geometry(1, 4, 4, 16, 16, 4, 0, tile, None) == nwg.NWG_EINVAL
        assert lib.nwg_last_status() == nwg.NWG_EINVAL
        assert lib.nwg_plan_geometry(16, 128, 128, 56, 56, 31, 15, tile, None) == nwg.NWG_EINVAL
        assert lib.nwg_plan_geometry_depthwise(1, 4, 16, 16, 4, 0, tile, None) == nwg.NWG_EINVAL
        assert lib.nwg_last_status() == nwg.NWG_EINVAL


def test_last_status_names_the_failure():
    lib = nwg.load_library()
    info = nwg.nwg_plan_info()
    assert lib.nwg_plan_geometry(0, 4, 4, 16, 16, 4, 0, 0, ctypes.byref(info)) == nwg.NWG_EINVAL
    assert lib.nwg_last_status() == nwg.NWG_EINVAL
    assert lib.nwg_plan_geometry(1, 4, 4, 99, 99, 32, 0, 0, ctypes.byref(info)) == \
        nwg.NWG_EUNSUPPORTED
    assert lib.nwg_last_status() == nwg.NWG_EUNSUPPORTED and b"depth" in lib.nwg_last_error()
    # maps of 2^31 values or more are refused before any size is formed
    assert lib.nwg_plan_geometry(1, 1, 1, 65536, 65536, 3, 1, 0, ctypes.byref(info)) == \
        nwg.NWG_EUNSUPPORTED


def test_tensor_checks_reject_bad_buffers_before_the_library():
    import torch
    from paper_2102_13272_amd.nwg import _ptr
    with pytest.raises(nwg.NwgError, match="float32"):
        _ptr(torch.zeros(16, dtype=torch.float64), 16, "x")
    with pytest.raises(nwg.NwgError, match="contiguous"):
        _ptr(torch.zeros(4, 8).t(), 32, "x")
    with pytest.raises(nwg.NwgError, match="elements"):
        _ptr(torch.zeros(15), 16, "y")
    with pytest.raises(nwg.NwgError, match="GPU"):
        _ptr(torch.zeros(16), 16, "w")
    with pytest.raises(nwg.NwgError, match="tensor"):
        _ptr(np.zeros(16, np.float32), 16, "w")


def test_no_silent_fallback_without_device():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(nwg.NwgError):
        nwg.Plan(1, 1, 1, 8, 8, 3)


@pytest.mark.parametrize("N", [1, 2, 3])
def test_fused_input_flag_and_workspace(N):
    # depth 3-4 with one or two output channels: nwg_conv2d fuses the input
    # transform into the contraction and the plan allocates no V
    for r in range(1, 32):
        g = nwg.plan_geometry(2, 4, N, 70, 66, r, (r - 1) // 2)
        fused = g["n"] in (3, 4) and N <= 2
        assert g["fused_input"] == int(fused), r
        if g["fused_conv"]:                     # one kernel x -> y: U only
            assert g["workspace_bytes"] == g["u_bytes"]
            continue
        v = 0 if fused else g["v_bytes"]
        assert g["workspace_bytes"] == g["u_bytes"] + v + g["yhat_bytes"]


@pytest.mark.parametrize("r", [1, 3, 7, 13, 31])
def test_depthwise_geometry(r):
    B, C, H, W, pad = 2, 6, 40, 33, (r - 1) // 2
    g = nwg.plan_geometry_depthwise(B, C, H, W, r, pad)
    d = nwg.plan_geometry(B, C, C, H, W, r, pad)
    assert g["depthwise"] == 1 and d["depthwise"] == 0
    for k in ("n", "Mn", "Ln", "th", "tw", "T", "P", "Ho", "Wo", "v_bytes", "yhat_bytes"):
        assert g[k] == d[k], k
    assert (g["M"], g["N"]) == (C, C)
    assert g["direct_flop"] == 2 * B * C * g["Ho"] * g["Wo"] * r * r
    if g["n"]:
        assert g["u_bytes"] == 4 * g["P"] * C
        assert g["ewmm_mults"] == g["P"] * g["T"] * C
        assert g["fused_input"] == int(g["n"] >= 3)
        z = g["yhat_bytes"] if g["n"] >= 3 else 0
        assert g["workspace_bytes"] == g["u_bytes"] + z
    else:
        assert g["u_bytes"] == 4 * C


def test_fused_conv_flag():
    # depth 1: M <= 8 and N <= 16; depth 2: M <= 2 and M N <= 64; depthwise depth 1-2
    for (M, N, r, want) in [(5, 5, 3, 1), (8, 16, 3, 1), (9, 4, 3, 0), (4, 17, 3, 0),
                            (1, 32, 5, 1), (2, 32, 5, 1), (2, 33, 5, 0), (3, 4, 5, 0),
                            (1, 1, 9, 0), (4, 4, 1, 0)]:
        g = nwg.plan_geometry(2, M, N, 40, 40, r, (r - 1) // 2)
        assert g["fused_conv"] == want, (M, N, r)
        if want:
            assert g["workspace_bytes"] == g["u_bytes"]
    for r, want in [(3, 1), (7, 1), (9, 0), (1, 0)]:
        g = nwg.plan_geometry_depthwise(2, 6, 40, 40, r, (r - 1) // 2)
        assert g["fused_conv"] == want, r


@pytest.mark.parametrize("r", list(range(1, 12)))
def test_f33_geometry_matches_oracle_levels(r):
    from oracle.nested import toom_cook_base
    B, M, N, H, W = 2, 3, 5, 40, 37
    pad = (r - 1) // 2
    tile = nwg.NWG_TILE_F3X3_3X3
    if r > 9:
        with pytest.raises(nwg.NwgError):
            nwg.plan_geometry(B, M, N, H, W, r, pad, tile)
        return
    g = nwg.plan_geometry(B, M, N, H, W, r, pad, tile)
    lv = nesting_levels(toom_cook_base(3, 3, [0, 1, -1, 2]), r)
    assert g["tile"] == tile
    assert g["n"] == lv.n and g["Mn"] == lv.Mn and g["Kn"] == lv.Kn
    assert g["strides"][:lv.n] == lv.strides
    if lv.n:
        assert (g["m"], g["rb"], g["l"], g["Ln"]) == (3, 3, 5, lv.Ln)
        P, T = 25 ** lv.n, B * g["th"] * g["tw"]
        assert g["P"] == P and g["T"] == T
        assert g["u_bytes"] == 4 * P * M * N and g["v_bytes"] == 4 * P * M * T
        assert g["yhat_bytes"] == 4 * (P // 25) * 15 * N * T
        assert g["workspace_bytes"] == g["u_bytes"] + g["v_bytes"] + g["yhat_bytes"]
    # never fused, even where the F(2x2,3x3) tile would be
    assert g["fused_input"] == 0 and g["fused_conv"] == 0 and g["pipeline_parts"] == 1
    with pytest.raises(nwg.NwgError):
        nwg.plan_geometry_depthwise(B, 4, H, W, r, pad, tile)


@pytest.mark.parametrize("shape,tile", [
    ((4, 32, 1, 256, 256, 9, 4), 1),      # one output channel at depth 2: fused F(3,3)
    ((4, 1, 32, 256, 256, 5, 2), 0),      # F(2,3) runs it in one kernel
    ((8, 64, 64, 56, 56, 9, 4), 1),       # depth 3 -> 2
    ((8, 64, 64, 56, 56, 7, 3), 0),       # same depth: F(2,3)
    ((8, 64, 64, 56, 56, 3, 1), 1),       # depth 1, wide channels
    ((4, 5, 5, 256, 256, 3, 1), 0),       # few channels
    ((16, 128, 128, 56, 56, 31, 15), 3),  # depth 4, wide channels: the mixed nest (5.07 / 1.90 ms)
    ((2, 16, 128, 56, 56, 31, 15), 0),    # depth 4, M < 32
    # depth 3 (r > 9) and 4 with M, N >= 32: the nest measured faster on
    # MI355X (ms per call, F(2,3) / mixed, one box) -- both skip their dead
    # groups, the mixed nest its dead points too, but it needs enough 12 x 12
    # or 36 x 36 tiles
    ((2, 128, 128, 56, 56, 31, 15), 0),   # 1.262 / 1.580 (8 tiles on the mixed nest)
    ((4, 128, 128, 28, 28, 31, 15), 0),   # 1.172 / 1.565 (4 tiles)
    ((1, 256, 256, 28, 28, 27, 13), 0),   # 2.77 / 5.42 (1 tile)
    ((16, 32, 32, 56, 56, 31, 15), 3),    # 0.889 / 0.457
    ((4, 64, 128, 112, 112, 23, 11), 3),  # 1.49 / 1.00
    ((1, 32, 32, 224, 224, 31, 15), 3),   # 0.81 / 0.43
    ((8, 64, 64, 56, 56, 17, 8), 3),      # 0.639 / 0.479
    ((32, 32, 64, 32, 32, 19, 9), 3),     # 0.381 / 0.286
    ((8, 64, 64, 56, 56, 13, 6), 3),      # depth 3: 0.238 / 0.190
    ((16, 128, 128, 56, 56, 13, 6), 3),   # 1.236 / 0.838
    ((16, 128, 128, 56, 56, 11, 5), 3),   # 0.838 / 0.587
    ((8, 64, 64, 56, 56, 15, 7), 0),      # 0.237 / 0.247 (r = 15: level-1 digit 3 live)
    ((4, 256, 256, 56, 56, 15, 7), 3),    # 1.310 / 1.136
    ((1, 32, 32, 64, 64, 1, 0), 0),       # 1x1
])
def test_auto_tile_choice(shape, tile):
    g = nwg.plan_geometry(*shape, tile=nwg.NWG_TILE_AUTO)
    assert g["tile"] == tile
    ref = nwg.plan_geometry(*shape, tile=tile)
    assert g == ref
    d = nwg.plan_geometry_depthwise(4, 16, 64, 64, 9, 4, tile=nwg.NWG_TILE_AUTO)
    assert d["tile"] == nwg.NWG_TILE_F2X2_3X3 and d["depthwise"] == 1


@pytest.mark.parametrize("r", [1, 2, 3, 4, 7, 9, 13, 31])
def test_ld_geometry_and_counts(r):
    from oracle.counts import ld_per_output
    B, M, N, H, W = 2, 3, 5, 40, 37
    pad = (r - 1) // 2
    g = nwg.plan_geometry(B, M, N, H, W, r, pad, nwg.NWG_TILE_LD_F2X2_3X3)
    c = -(-r // 3)
    Ho, Wo = H + 2 * pad - r + 1, W + 2 * pad - r + 1
    assert g["tile"] == nwg.NWG_TILE_LD_F2X2_3X3 and g["ld_c"] == c
    assert (g["n"], g["P"], g["Mn"], g["Kn"], g["Ln"]) == (1, 16, 2, 3 * c, 3 * c + 1)
    assert (g["th"], g["tw"]) == (-(-Ho // 2), -(-Wo // 2))
    T = B * g["th"] * g["tw"]
    assert g["T"] == T
    assert g["u_bytes"] == 4 * 16 * M * c * c * N and g["v_bytes"] == 4 * 16 * M * c * c * T
    assert g["yhat_bytes"] == 4 * 4 * N * T
    # Sec. II.B's count, (l/m)^2 ceil(R/r)^2 multiplications per output and channel pair
    per_out = ld_per_output(2, 3, r)
    assert g["ewmm_mults"] == per_out * (T * 4) * M * N
    assert g["fused_input"] == 0 and g["fused_conv"] == 0


def test_ld_multiplications_match_the_oracle_loop():
    from oracle.lindecomp import ld_conv2d
    from oracle.nested import MultCounter
    rng = np.random.default_rng(0)
    B, M, N, H, W, r, pad = 1, 2, 3, 9, 8, 5, 2
    x = rng.standard_normal((B, M, H, W))
    w = rng.standard_normal((N, M, r, r))
    cnt = MultCounter()
    ld_conv2d(x, w, pad, counter=cnt)
    g = nwg.plan_geometry(B, M, N, H, W, r, pad, nwg.NWG_TILE_LD_F2X2_3X3)
    assert g["ewmm_mults"] == cnt.count


def test_ld_workspace_holds_the_k_slices():
    # C3-shaped layer: 7 x 1 column tiles, so the M c^2 = 1600 channels are
    # cut into slices whose partial Z the plan holds
    g = nwg.plan_geometry(8, 64, 64, 56, 56, 13, 6, nwg.NWG_TILE_LD_F2X2_3X3)
    parts = (g["workspace_bytes"] - g["u_bytes"] - g["v_bytes"]) // g["yhat_bytes"]
    assert parts > 1 and (64 * 25 // 32) % parts == 0
    assert g["workspace_bytes"] == g["u_bytes"] + g["v_bytes"] + parts * g["yhat_bytes"]


@pytest.mark.parametrize("r", [1, 3, 5, 7, 8, 9, 13, 15, 16, 23, 31, 39, 40])
def test_mixed_geometry_matches_oracle_chain(r):
    """NWG_TILE_MIX_F23_F33: the library's recurrence with F(2,3) at levels 1-2
    and F(3,3) above equals the oracle's mixed-chain levels (oracle.mixed)."""
    from oracle.mixed import mixed_levels, mults_per_output
    from oracle.nested import toom_cook_base
    B, M, N, H, W = 2, 3, 5, 80, 77
    pad = (r - 1) // 2
    tile = nwg.NWG_TILE_MIX_F23_F33
    if r > 39:
        with pytest.raises(nwg.NwgError):
            nwg.plan_geometry(B, M, N, H, W, r, pad, tile)
        return
    g = nwg.plan_geometry(B, M, N, H, W, r, pad, tile)
    if r <= 7:        # only the two F(2,3) levels: the F(2x2,3x3) plan
        assert g == nwg.plan_geometry(B, M, N, H, W, r, pad)
        assert g["tile"] == nwg.NWG_TILE_F2X2_3X3 and g["outer33"] == 0
        return
    f23, f33 = base_f23(), toom_cook_base(3, 3, [0, 1, -1, 2])
    lv = mixed_levels([f23, f23, f33, f33], r)
    assert g["tile"] == tile and g["outer33"] == lv.n - 2
    assert g["n"] == lv.n and g["Mn"] == lv.Mn and g["Kn"] == lv.Kn and g["Ln"] == lv.Ln
    assert g["strides"] == lv.strides
    assert (g["m"], g["rb"], g["l"]) == (2, 3, 4)
    P, T = lv.P1 ** 2, B * g["th"] * g["tw"]
    assert g["P"] == P and g["T"] == T
    assert g["th"] == -(-(H + 2 * pad - r + 1) // lv.Mn)
    assert g["u_bytes"] == 4 * P * M * N and g["v_bytes"] == 4 * P * M * T
    assert g["yhat_bytes"] == 4 * (P // 4) * N * T
    # depth 4: scratch for the level-4 input blocks (26 x 26 per branch, tile
    # and channel) and the level-3 output blocks (12 x 12 per branch, tile
    # and channel), used in turn
    scratch = 4 * max(25 * 676 * M * T, 25 * 144 * N * T) if lv.n == 4 else 0
    assert g["workspace_bytes"] == g["u_bytes"] + g["v_bytes"] + g["yhat_bytes"] + scratch
    assert g["ewmm_mults"] == P * T * M * N
    # per output and channel pair: prod l_j^2 / M_n^2, the oracle's count
    assert mults_per_output([f23, f23, f33, f33], r) == \
        __import__("fractions").Fraction(P, lv.Mn ** 2)
    assert g["fused_input"] == 0 and g["fused_conv"] == 0 and g["fused_output"] == 0
    # one output channel would take the fused kernel on the F(2x2,3x3) tile
    g1 = nwg.plan_geometry(B, M, 1, H, W, r, pad, tile)
    assert g1["fused_input"] == 0
    with pytest.raises(nwg.NwgError):
        nwg.plan_geometry_depthwise(B, 4, H, W, r, pad, tile)


def test_mixed_geometry_of_the_31x31_workload():
    g = nwg.plan_geometry(16, 128, 128, 56, 56, 31, 15, nwg.NWG_TILE_MIX_F23_F33)
    assert (g["n"], g["Mn"], g["Kn"], g["Ln"], g["P"]) == (4, 36, 39, 74, 160000)
    assert (g["th"], g["tw"], g["T"]) == (2, 2, 64)
    # 1.64x fewer contraction FLOPs than four F(2,3) levels (65536 points x 256 tiles)
    f23 = nwg.plan_geometry(16, 128, 128, 56, 56, 31, 15)
    assert f23["P"] * f23["T"] / (g["P"] * g["T"]) == pytest.approx(1.6384)


def _oracle_live_prefixes(r, tile=nwg.NWG_TILE_MIX_F23_F33):
    """Digit prefixes (q_n .. q_2, the outermost most significant) of the
    mixed chain (or the chain of F(2,3) levels) at kernel size r with a point
    whose row of the oracle's kernel-transform matrix is nonzero over the r
    real taps."""
    from oracle.mixed import mixed_levels, kernel_matrix, _digits
    from oracle.nested import toom_cook_base
    f23, f33 = base_f23(), toom_cook_base(3, 3, [0, 1, -1, 2])
    n = nwg.plan_geometry(1, 1, 1, 64, 64, r, 0, tile)["n"]
    up = f33 if tile == nwg.NWG_TILE_MIX_F23_F33 else f23
    lv = mixed_levels([f23, f23] + [up] * (n - 2), r)
    KG = kernel_matrix(lv)
    rad = [b.l for b in lv.bases]                 # level 1 .. n
    live, q1 = set(), set()
    for p in range(lv.P1):
        d = _digits(p, rad)                       # (q_1, ..., q_n), q_1 most significant
        if any(KG[p, k] != 0 for k in range(r)):
            idx = 0
            for j in range(n - 1, 0, -1):         # q_n first
                idx = idx * rad[j] + d[j]
            live.add(idx)
            q1.add(d[0])
    npref = 1
    for j in range(1, n):
        npref *= rad[j]
    return live, npref, q1


@pytest.mark.parametrize("r", [8, 9, 12, 13, 15, 16, 17, 24, 27, 31, 33, 35, 38, 39])
def test_mixed_live_groups_are_the_oracle_kernel_rows_that_reach_a_real_tap(r):
    """The library skips the mixed nest's groups whose transformed kernel is zero
    for every w; its per-axis prefix mask must be the set of prefixes with a
    nonzero row in the oracle's kernel-transform matrix (Sec. III.B's
    reordering and G^(x)n, written independently)."""
    g = nwg.plan_geometry(2, 8, 8, 64, 64, r, r // 2, nwg.NWG_TILE_MIX_F23_F33)
    live, npref, q1 = _oracle_live_prefixes(r)
    # level-1 digits: the library skips digit 3 exactly when no point with it
    # has a nonzero kernel row (r below the nest's 39 or 15 taps)
    assert g["level1_live"] == sum(1 << q for q in q1)
    assert (g["level1_live"] == 0x7) == (r < g["Kn"])
    if g["live_np"] == 0:
        assert len(live) == npref and g["live_groups"] == g["P"] // 16
        return
    mask = g["live_prefix"][0] | (g["live_prefix"][1] << 64)
    lib = {i for i in range(npref) if (mask >> i) & 1}
    assert lib == live
    assert g["live_np"] == len(live) and g["live_groups"] == len(live) ** 2


@pytest.mark.parametrize("r", [5, 6, 7, 8, 9, 11, 13, 15, 16, 17, 20, 23, 29, 31])
def test_f23_chain_live_groups_are_the_oracle_kernel_rows_that_reach_a_real_tap(r):
    """Unfused dense chains of F(2x2,3x3) levels (depth 3 and 4) skip the
    groups whose transformed kernel is zero for every w; the prefix mask must
    be the set of prefixes with a nonzero row of the oracle's kernel-transform
    matrix, and every level-1 digit stays (F(2,3) chains skip groups only)."""
    g = nwg.plan_geometry(2, 8, 8, 64, 64, r, r // 2)
    assert g["tile"] == nwg.NWG_TILE_F2X2_3X3 and g["level1_live"] == 0xf
    if g["n"] < 3 or g["fused_conv"] or g["fused_input"] or g["fused_output"]:
        assert g["live_np"] == 0 and g["live_groups"] == g["P"] // 16
        return
    live, npref, _ = _oracle_live_prefixes(r, nwg.NWG_TILE_F2X2_3X3)
    if g["live_np"] == 0:
        assert len(live) == npref and g["live_groups"] == g["P"] // 16
        return
    mask = g["live_prefix"][0] | (g["live_prefix"][1] << 64)
    lib = {i for i in range(npref) if (mask >> i) & 1}
    assert lib == live
    assert g["live_np"] == len(live) and g["live_groups"] == len(live) ** 2
