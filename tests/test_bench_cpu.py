"""Host logic of bench.py, without a GPU: the one-GPU guard, the algorithmic
bytes and FLOPs the roofline divides by, and the conversion of rocprofv3
FETCH_SIZE / WRITE_SIZE counters into HBM bytes per launch (scaled by a copy
kernel of known size, summed over a stage's kernels, and reported only while
the kernel sources are unchanged)."""
import csv
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
from paper_2102_13272_amd import nwg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU only" in p.stderr and p.stdout == ""


@pytest.mark.parametrize("tile", [nwg.NWG_TILE_F2X2_3X3, nwg.NWG_TILE_MIX_F23_F33])
def test_stage_bytes_are_the_plan_buffers_and_the_layer_tensors(tile):
    # the 31 x 31 layer: B = 16, 128 -> 128, 56 x 56, 'same' padding
    B, M, N, H, W, r, pad = 16, 128, 128, 56, 56, 31, 15
    g = nwg.plan_geometry(B, M, N, H, W, r, pad, tile)
    sb = bench.stage_bytes_flops(g)
    x, y, w = 4 * B * M * H * W, 4 * B * N * H * W, 4 * N * M * r * r
    # the contraction moves 4 bytes per U and V value once, and one Z value
    # per four points (the level-1 output fold), over the groups it computes,
    # the live ones (a tap reaches them): on four F(2x2,3x3) levels 54^2 of
    # 64^2, every point of each multiplied; on the mixed nest 72^2 of 100^2,
    # three of their four quads (level-1 row digit 3 is dead at r = 31), and
    # 3 x 3 of their 16 points multiplied
    mix = tile == nwg.NWG_TILE_MIX_F23_F33
    G, npt = g["live_groups"], 9 if mix else 16
    assert G == (72 * 72 if mix else 54 * 54) and g["P"] // 16 == (100 * 100 if mix else 64 * 64)
    assert g["level1_live"] == (0x7 if mix else 0xf) and g["mix_planar"] == int(mix)
    # the mixed nest's planar U and V hold the 9 live points of each live
    # group; the F(2,3) plan's U and V hold every group, its kernel transform
    # writes them all and its input transform the live groups' V
    Ga = G if mix else g["P"] // 16
    U, V = 4 * npt * Ga * M * N, 4 * npt * Ga * M * g["T"]
    Uc, Vc, Z = 4 * npt * G * M * N, 4 * npt * G * M * g["T"], 4 * 4 * G * N * g["T"]
    assert (g["u_bytes"], g["v_bytes"], g["yhat_bytes"]) == (
        U, V, 4 * (g["P"] // 4) * N * g["T"])
    assert sb["kernel_transform"] == (w + U, 0.0)
    assert sb["input_transform"] == (x + Vc, 0.0)
    assert sb["output_transform"] == (Z + y, 0.0)
    b, f = sb["contraction"]
    assert b == Uc + Vc + Z and f == g["contract_flop"] == 2.0 * npt * G * M * N * g["T"]


def test_depth0_stage_bytes_are_a_channel_gemm():
    g = nwg.plan_geometry(2, 8, 4, 10, 12, 1, 0)
    sb = bench.stage_bytes_flops(g)
    assert set(sb) == {"kernel_transform", "contraction"}
    x, y = 4 * 2 * 8 * 10 * 12, 4 * 2 * 4 * 10 * 12
    assert sb["contraction"] == (x + y + 4 * 8 * 4, 2.0 * 2 * 4 * 8 * 10 * 12)


def _counter_csv(path, counter, rows):
    with open(path, "w", newline="") as fh:
        wr = csv.DictWriter(fh, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        wr.writeheader()
        for name, kib in rows:
            wr.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": kib})


def test_traffic_is_scaled_by_the_copy_and_summed_per_stage(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (tmp_path / "profiles").mkdir()
    copy = "__amd_rocclr_copyBuffer"
    l4 = "nwg::(anonymous namespace)::input_mix_l4(float const*, float*, int)"
    l3 = "void nwg::(anonymous namespace)::input_xform_mix<2>(float const*, float*)"
    ct = "void nwg::(anonymous namespace)::contract_deep_persist<128, 64>(float4 const*)"
    # 1 MiB copy: FETCH_SIZE reads half the bytes, WRITE_SIZE all of them
    _counter_csv(tmp_path / "f.csv", "FETCH_SIZE",
                 [(copy, 512.0), (l4, 100.0), (l4, 300.0), (l3, 50.0), (ct, 1000.0)])
    _counter_csv(tmp_path / "w.csv", "WRITE_SIZE",
                 [(copy, 1024.0), (l4, 10.0), (l4, 30.0), (l3, 5.0), (ct, 40.0)])
    out = bench.traffic_from_counters("wl", "auto", str(tmp_path / "f.csv"),
                                      str(tmp_path / "w.csv"), 1)
    assert out["fetch_scale"] == 2.0 and out["write_scale"] == 1.0
    k = out["kernels"]
    # input transform: the level-4 kernel (mean of its two dispatches) plus
    # the level-3 kernel
    assert k["input_transform"]["fetch_bytes"] == (200 + 50) * 1024 * 2
    assert k["input_transform"]["write_bytes"] == (20 + 5) * 1024
    assert k["input_transform"]["kernel"] == "input_mix_l4 + input_xform_mix<2>"
    assert k["contraction"]["hbm_bytes_per_launch"] == 1000 * 1024 * 2 + 40 * 1024
    with open(tmp_path / "profiles" / "traffic_wl_auto.json") as fh:
        assert json.load(fh) == out
    # read back while the sources are unchanged, for the same tile only
    assert bench.measured_traffic("wl", "contraction", "auto") == 1000 * 1024 * 2 + 40 * 1024
    assert bench.measured_traffic("wl", "contraction", "f23") is None
    assert bench.measured_traffic("other", "contraction", "auto") is None
    # a stale hash (the kernel changed since the counters were taken) reads as unmeasured
    out["kernels"]["contraction"]["source_hash"] = "0" * 16
    with open(tmp_path / "profiles" / "traffic_wl_auto.json", "w") as fh:
        json.dump(out, fh)
    assert bench.measured_traffic("wl", "contraction", "auto") is None


def test_traffic_needs_the_copy_calibration(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    _counter_csv(tmp_path / "f.csv", "FETCH_SIZE", [("contract_x", 1.0)])
    _counter_csv(tmp_path / "w.csv", "WRITE_SIZE", [("contract_x", 1.0)])
    with pytest.raises(SystemExit):
        bench.traffic_from_counters("wl", "auto", str(tmp_path / "f.csv"),
                                    str(tmp_path / "w.csv"), 1)


def test_committed_traffic_summaries_match_the_current_contraction_source():
    """The default line's traffic comes from profiles/traffic_c5_r31_auto.json;
    its contraction entry must be the one taken on the current kernel source."""
    for wl, tile in (("c5_r31", "auto"), ("c5_r31", "f23"), ("c3_r13", "auto")):
        t = bench.measured_traffic(wl, "contraction", tile)
        assert t is not None and t > 0


def test_cpu_baseline_reports_parity_of_the_outputs_it_is_given():
    """The oracle leg times whole images and compares every GPU output of the
    same run on those images; a perturbation beyond the fp32 bar fails."""
    from oracle.direct import direct_conv2d
    from paper_2102_13272_amd.workloads import WORKLOADS, make_workload
    x, (w,) = make_workload("c1_r4_valid")
    y = direct_conv2d(x, w, WORKLOADS["c1_r4_valid"].layers[0].pad).astype(np.float32)
    bad = y.copy()
    bad[0, 1, 2, 3] += 0.01 * np.abs(y).max()
    base, par = bench.cpu_baseline("c1_r4_valid", 0.0, {"good": y, "bad": bad})
    assert base["kind"] == "oracle" and base["sample"].startswith("1 of 1 images")
    assert base["cores"] >= 1 and base["host_nproc"] >= 1
    assert par["good"]["ok"] and par["good"]["rel_l2"] < 1e-6
    assert not par["bad"]["ok"] and par["bad"]["max_abs_over_max"] > 1e-3
    assert par["good"]["outputs"] == y.size


def test_kernel_transform_entry_is_its_bytes_over_its_time():
    # the mixed nest's 31 x 31 layer: w (63 MB) + the planar U (the 9 live
    # points of 5184 live groups of 10000: 3.06 GB) in 2.25 ms
    g = nwg.plan_geometry(16, 128, 128, 56, 56, 31, 15, nwg.NWG_TILE_MIX_F23_F33)
    nbytes = bench.stage_bytes_flops(g)["kernel_transform"][0]
    e = bench.kernel_transform_entry(2.25, nbytes)
    assert e["bytes"] == 4 * 128 * 128 * 31 * 31 + 4 * 9 * 5184 * 128 * 128
    assert e["GB_s"] == pytest.approx(nbytes / 2.25e-3 / 1e9, rel=1e-3)
    assert e["hbm_frac"] == pytest.approx(e["GB_s"] / bench.PEAK_HBM_GBS, rel=1e-3)
    assert e["bound"] == "hbm" and e["ms_once"] == 2.25
    assert bench.kernel_transform_entry(0.0, nbytes)["GB_s"] == 0.0
