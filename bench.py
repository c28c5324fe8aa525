#!/usr/bin/env python3
"""Benchmark: nested-Winograd convolution on one MI355X.

A step is one pass of the whole hot path (input transform, per-point channel
contraction, output transform -- every layer of the workload) over one batch
of synthetic input already resident in HBM.  The kernel transform runs once
per weight set during warm-up (the plan caches U); its time is reported
separately and in `value_incl_kernel_transform`.

Prints ONE JSON line.  `value` is direct-convolution-equivalent TFLOP/s
(2*B*N*M*Ho*Wo*r^2 per layer, summed, divided by the step time).  The
roofline object describes the kernel with the largest share of the step,
with its algorithmic bytes or FLOPs and its average duration from HIP
events the library records on the stream it launches on.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, GB/s
PEAK_FP32_MFMA_TFLOPS = 157.3  # MI355X dense fp32 matrix
PEAK_BF16_MFMA_TFLOPS = 2500.0  # MI355X dense bf16 matrix
METRIC = "direct-conv-equiv TFLOP/s & fraction of fp32 MFMA/HBM roofline, 1 MI355X"
STAGES = ["kernel_transform", "input_transform", "contraction", "output_transform"]
NWG_TILE_MIX = 3               # the mixed F(2,3)/F(3,3) nest (include/nwg.h)
CSRC = os.path.join(ROOT, "paper_2102_13272_amd", "csrc")


def stage_bytes_flops(info: dict):
    """Algorithmic bytes (fp32) and FLOPs per launch of each stage of one layer."""
    P, M, N, T = info["P"], info["M"], info["N"], info["T"]
    B, H, W, Ho, Wo, r = info["B"], info["H"], info["W"], info["Ho"], info["Wo"], info["r"]
    dw = bool(info.get("depthwise"))
    mk = 1 if dw else M                      # input channels per kernel
    x = 4 * B * M * H * W
    y = 4 * B * N * Ho * Wo
    w = 4 * N * mk * r * r
    flop = info["contract_flop"]
    if info["n"] == 0:
        return {"kernel_transform": (w + 4 * mk * N, 0.0),
                "contraction": (x + y + 4 * mk * N, flop)}
    # Z: the contraction's output after (part of) the first output level: P/4
    # values per (n, t) on F(2x2,3x3), 3P/5 on F(3x3,3x3) (the plan's yhat_bytes)
    U, V, Yh = info["u_bytes"], info["v_bytes"], info["yhat_bytes"]
    if info.get("tile") == NWG_TILE_MIX and info["n"] >= 3:
        # the mixed nest moves only its live groups' U, V and Z; of U and V
        # the planar layout holds just the 3 x 3 live points of a group, the
        # quad layout the quads whose level-1 row digit is live (3 of 4 when
        # digit 3 is dead, each float4 still carrying its dead fourth point)
        G, live = P // 16, info["live_groups"]
        nq = 3 if info.get("level1_live") == 0x7 else 4
        if not info.get("mix_planar"):      # planar: U and V hold the live points only
            U, V = U // G * live * nq // 4, V // G * live * nq // 4
        Yh = Yh // G * live
    # a dense F(2x2,3x3) chain with dead groups: the kernel transform writes
    # every group, the input transform the live ones (while a wavefront's
    # four level-3 branches of V span at most 2^30 bytes), the contraction
    # reads and writes the live ones only, and the output transform reads
    # only their Z
    Uc, Vc, Zc, Vw = U, V, Yh, V
    if (info.get("tile") == 0 and not dw and info["n"] >= 3 and info.get("live_np", 0) > 0
            and not (info.get("fused_input") or info.get("fused_conv") or info.get("fused_output"))):
        G, live = P // 16, info["live_groups"]
        Uc, Vc, Zc = U // G * live, V // G * live, Yh // G * live
        if 256 * info["M"] * info["T"] * 16 <= 1 << 30:
            Vw = Vc
    if info.get("fused_output"):
        # input transform, then the output transform that forms the contraction
        return {"kernel_transform": (w + U, 0.0), "input_transform": (x + V, 0.0),
                "contraction": (U + V + y, flop)}
    if info.get("fused_conv"):
        # one kernel: x and U in, y out
        return {"kernel_transform": (w + U, 0.0), "contraction": (x + U + y, flop)}
    if info.get("fused_input"):
        # one kernel reads x and U and writes Z; V never reaches memory
        return {"kernel_transform": (w + U, 0.0),
                "contraction": (x + U + Yh, flop),
                "output_transform": (Yh + y, 0.0)}
    return {"kernel_transform": (w + U, 0.0),
            "input_transform": (x + Vw, 0.0),
            "contraction": (Uc + Vc + Zc, flop),
            "output_transform": (Zc + y, 0.0)}


def source_hash(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {"input_transform": ["input_xform.hip", "mixed.hip", "nwg_internal.h"],
                  "contraction": ["contract_mfma.hip", "nwg_internal.h"],
                  "output_transform": ["output_xform.hip", "mixed.hip", "nwg_internal.h"],
                  "kernel_transform": ["kernel_xform.hip", "mixed.hip", "nwg_internal.h"]}


def measured_traffic(workload: str, stage: str, tile: str):
    """HBM bytes per launch from a committed rocprofv3 counter summary, if it
    was taken on the current kernel source with the same --tile; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}_{tile}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        d = json.load(fh)
    ent = d.get("kernels", {}).get(stage)
    if d.get("tile", "f23") != tile:
        return None
    if not ent or ent.get("source_hash") != source_hash(KERNEL_SOURCES[stage]):
        return None
    return ent.get("hbm_bytes_per_launch")


STAGE_OF_KERNEL = [("contract", "contraction"), ("gemm_mfma", "contraction"),
                   ("input_xform", "input_transform"), ("input_mix", "input_transform"),
                   ("output_xform", "output_transform"), ("kernel_xform", "kernel_transform")]


def traffic_from_counters(workload: str, tile: str, fetch_csv: str, write_csv: str,
                          copy_mib: int):
    """HBM bytes per launch of each stage from two rocprofv3 --pmc runs.

    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are scaled by what the same
    counters read for the plain device-to-device copy of `copy_mib` MiB that
    `--calibrate-copy-mib` performs at the start of the profiled run.
    A stage that runs several kernels (the mixed nest's input and output
    transforms) gets their sum.  Writes profiles/traffic_<workload>_<tile>.json
    and returns its content.
    """
    import csv
    from collections import defaultdict

    def per_kernel(path, counter):
        vals = defaultdict(list)
        with open(path) as fh:
            for row in csv.DictReader(fh):
                if row["Counter_Name"] == counter:
                    vals[row["Kernel_Name"]].append(float(row["Counter_Value"]))
        return vals

    fetch, write = per_kernel(fetch_csv, "FETCH_SIZE"), per_kernel(write_csv, "WRITE_SIZE")
    copy_bytes = copy_mib * (1 << 20)
    cf = [v for k, v in fetch.items() if "copyBuffer" in k]
    cw = [v for k, v in write.items() if "copyBuffer" in k]
    if not cf or not cw:
        raise SystemExit("no copy-kernel dispatch in the counter files (run with --calibrate-copy-mib)")
    fscale = copy_bytes / (cf[0][0] * 1024.0)
    wscale = copy_bytes / (cw[0][0] * 1024.0)
    out = {"workload": workload, "tile": tile, "copy_calibration_bytes": copy_bytes,
           "fetch_scale": round(fscale, 4), "write_scale": round(wscale, 4), "kernels": {}}
    for name in fetch:
        stage = next((st for key, st in STAGE_OF_KERNEL if key in name), None)
        if stage is None or name not in write:
            continue
        f = sum(fetch[name]) / len(fetch[name]) * 1024.0 * fscale
        w = sum(write[name]) / len(write[name]) * 1024.0 * wscale
        short = name.split("::")[-1].split("(")[0] if "(anonymous namespace)::" in name else name
        short = name.split("(anonymous namespace)::")[-1].split("(")[0] if "(anonymous namespace)::" in name else short
        ent = out["kernels"].setdefault(stage, {"kernel": "", "dispatches": len(fetch[name]),
                                                "fetch_bytes": 0, "write_bytes": 0,
                                                "hbm_bytes_per_launch": 0,
                                                "source_hash": source_hash(KERNEL_SOURCES[stage])})
        ent["kernel"] = (ent["kernel"] + " + " if ent["kernel"] else "") + short[:120]
        ent["fetch_bytes"] += round(f)
        ent["write_bytes"] += round(w)
        ent["hbm_bytes_per_launch"] += round(f + w)
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}_{tile}.json")
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)
    return out


def blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        return max([d.get("num_threads", 1) for d in threadpool_info()
                    if d.get("user_api") == "blas"] or [1])
    except Exception:
        return os.cpu_count() or 1


def host_cores() -> dict:
    """The host's logical CPUs (os.cpu_count, like nproc without a mask) and
    the ones this process may run on (sched_getaffinity, what nproc prints)."""
    try:
        usable = len(os.sched_getaffinity(0))
    except Exception:
        usable = os.cpu_count() or 1
    return {"cpu_count": os.cpu_count() or 1, "nproc": usable}


REL_L2, MAX_ABS_FRAC = 1e-4, 1e-3     # the fp32 bar against the fp64 oracle


def cpu_baseline(workload: str, target_s: float, outputs=None):
    """The fp64 oracle timed on this host's cores over a bounded sample of the
    workload (whole images, all channels, every layer), and the parity of the
    GPU outputs of the same run (a dict of name -> numpy [B][N][Ho][Wo] of the
    last layer) on the sampled images: rel-L2 and max-abs over all their
    outputs, against the fp32 bar.  Returns (baseline, {name: parity})."""
    from oracle.direct import direct_conv2d, direct_depthwise_conv2d
    from paper_2102_13272_amd.workloads import WORKLOADS, make_workload

    def conv(L, xs, w):
        return (direct_depthwise_conv2d if L.depthwise else direct_conv2d)(xs, w, L.pad)
    wl = WORKLOADS[workload]
    x, ws = make_workload(workload)
    B = wl.layers[0].B
    flop = 0.0
    refs = []
    t0 = time.perf_counter()
    for b in range(B):
        cur = x[b:b + 1].astype(np.float64)
        for L, w in zip(wl.layers, ws):
            cur = conv(L, cur, w)
            flop += L.direct_flop / L.B
        refs.append(cur[0])
        if time.perf_counter() - t0 >= target_s:
            break
    dt = time.perf_counter() - t0
    images = len(refs)
    what = "all channels" if len(wl.layers) == 1 else f"through all {len(wl.layers)} layers"
    base = {"value": flop / dt / 1e12, "unit": "TFLOP/s", "cores": blas_threads(), "kind": "oracle",
            "sample": f"{images} of {B} images of the workload, {what}",
            "seconds": round(dt, 3), **{"host_" + k: v for k, v in host_cores().items()}}
    ref = np.stack(refs)
    den = np.linalg.norm(ref)
    scale = float(np.abs(ref).max())
    parity = {}
    for key, y in (outputs or {}).items():
        got = np.asarray(y[:images], dtype=np.float64)
        rel = float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))
        mabs = float(np.abs(got - ref).max())
        ok = bool(np.isfinite(got).all() and rel <= REL_L2 and mabs <= MAX_ABS_FRAC * scale)
        parity[key] = {"rel_l2": rel, "max_abs_over_max": mabs / scale if scale else mabs,
                       "images": images, "outputs": int(ref.size), "ok": ok,
                       "bar": {"rel_l2": REL_L2, "max_abs_over_max": MAX_ABS_FRAC},
                       "oracle": "fp64 direct correlation"}
    return base, parity


TILE_NAMES = {0: "F(2x2,3x3)", 1: "F(3x3,3x3)", 2: "linear decomposition on F(2x2,3x3)",
              3: "mixed F(2,3)/F(3,3) nest"}


def run_workload(torch, nwg, name: str, tile: str, precision: str, steps: int, warmup: int,
                 pipeline_parts: int = 0, graph: bool = False) -> dict:
    """Plans for every layer of the workload, warm-up (which transforms the
    weights once), K timed steps with the library's per-stage events off, then
    K more with them on for the per-stage times.  Returns the measurements, the
    plans (open) and the last layer's output tensor of the timed run."""
    from paper_2102_13272_amd.workloads import WORKLOADS, make_workload
    wl = WORKLOADS[name]
    x, ws = make_workload(name)
    xd = torch.from_numpy(x).to("cuda")
    wds = [torch.from_numpy(w).to("cuda") for w in ws]

    def tile_for(L):
        if tile == "auto":
            return nwg.NWG_TILE_AUTO
        if tile == "f33" and not L.depthwise and L.r <= 9:
            return nwg.NWG_TILE_F3X3_3X3
        if tile == "ld" and not L.depthwise and L.r > 1:
            return nwg.NWG_TILE_LD_F2X2_3X3
        if tile == "mix" and not L.depthwise and L.r >= 8:
            return nwg.NWG_TILE_MIX_F23_F33
        return nwg.NWG_TILE_F2X2_3X3

    plans = [nwg.Plan(L.B, L.M, L.N, L.H, L.W, L.r, L.pad, tile=tile_for(L),
                      depthwise=L.depthwise) for L in wl.layers]
    if pipeline_parts:
        for p in plans:
            if p.info["pipeline_parts"] > 1 or pipeline_parts == 1:
                p.set_pipeline(pipeline_parts)
    if precision == "bf16_split":
        for p in plans:
            try:
                p.set_precision(nwg.NWG_PRECISION_BF16_SPLIT)
            except nwg.NwgError:
                pass            # this layer keeps fp32
    outs = [torch.empty(p.y_shape, dtype=torch.float32, device="cuda") for p in plans]
    stream = torch.cuda.current_stream()

    def step(s=None):
        cur = xd
        for p, w, y in zip(plans, wds, outs):
            p.conv2d(cur, w, y, s or stream)
            cur = y

    # warm-up (includes the one kernel transform per layer), then timed steps
    for p in plans:
        p.set_timing(True)
    for _ in range(max(1, warmup)):
        step()
    torch.cuda.synchronize()
    warm = [p.get_timing() for p in plans]
    kx_first_ms = sum(ms[0] for ms, _ in warm)
    # steady-state kernel transform: the first call above also pays the lazy
    # load of the code objects; time 3 more calls per layer into a spare U
    kx_ms = 0.0
    for p, w, ms in zip(plans, wds, (m for m, _ in warm)):
        try:
            U2 = torch.empty(p.u_shape, dtype=torch.float32, device="cuda")
            p.kernel_transform(w, U2, stream)
            k0, k1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            k0.record(stream)
            for _ in range(3):
                p.kernel_transform(w, U2, stream)
            k1.record(stream)
            torch.cuda.synchronize()
            kx_ms += k0.elapsed_time(k1) / 3
            del U2
        except nwg.NwgError:
            kx_ms += ms[0]      # no stage call (depth 0, depthwise): first call
    # its algorithmic bytes (w read, U written), summed over layers
    kx_bytes = float(sum(stage_bytes_flops(p.info)["kernel_transform"][0] for p in plans))

    # the timed steps run with the library's per-stage events off (recording
    # them puts work between the launches); a second pass of K steps with
    # them on gives the per-stage times
    for p in plans:
        p.set_timing(False)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / steps
    y_timed = outs[-1].cpu().numpy()
    for p in plans:
        p.set_timing(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    timing = [p.get_timing() for p in plans]
    for p in plans:
        p.set_timing(False)
    ms_step_eager = ms_step
    if graph:
        # one step captured (weights already transformed, timing off: the
        # captured work is exactly the step's kernels), then K replays timed
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap):
            step(torch.cuda.current_stream())
        g.replay()
        torch.cuda.synchronize()
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for _ in range(steps):
            g.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        ms_step = g0.elapsed_time(g1) / steps

    direct_flop = float(sum(L.direct_flop for L in wl.layers))
    # per-stage accounting summed over layers
    stages = {}
    for p, (ms, cnt) in zip(plans, timing):
        bf = stage_bytes_flops(p.info)
        parts = p.info["pipeline_parts"]
        for si, sname in enumerate(STAGES):
            if sname == "kernel_transform" or cnt[si] == 0:
                continue
            b, f = bf[sname]
            if sname in ("input_transform", "contraction") and parts > 1:
                # the two-stream pipeline launches these in `parts` pieces
                b, f = b / parts, f / parts
            st = stages.setdefault(sname, {"ms_total": 0.0, "launches": 0, "bytes": 0.0,
                                           "flop": 0.0, "per_layer": []})
            st["ms_total"] += ms[si]
            st["launches"] += cnt[si]
            st["bytes"] += b * cnt[si]
            st["flop"] += f * cnt[si]
            st["per_layer"].append({"r": p.info["r"], "n": p.info["n"],
                                    "avg_us": round(1e3 * ms[si] / cnt[si], 2),
                                    **({"pieces": parts} if parts > 1 and sname in (
                                        "input_transform", "contraction") else {}),
                                    **({"fused_input": True} if p.info["fused_input"]
                                       and sname == "contraction" else {}),
                                    **({"fused_conv": True} if p.info["fused_conv"]
                                       and sname == "contraction" else {})})
    # split precision: the MFMAs run on bf16 and execute 4 partial products
    # per algorithmic multiply-add
    split = any(p.info["precision"] == nwg.NWG_PRECISION_BF16_SPLIT for p in plans)
    peak_mm = PEAK_BF16_MFMA_TFLOPS if split else PEAK_FP32_MFMA_TFLOPS
    flop_x = 4.0 if split else 1.0
    detail = {}
    for sname, st in stages.items():
        sec = st["ms_total"] * 1e-3
        gbs = st["bytes"] / sec / 1e9
        tfs = st["flop"] / sec / 1e12
        detail[sname] = {"ms_per_step": round(st["ms_total"] / steps, 4),
                         "launches_per_step": st["launches"] // steps,
                         "GB_s": round(gbs, 1), "hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
                         "TFLOP_s": round(tfs, 2),
                         "mfma_frac": round(flop_x * tfs / peak_mm, 4),
                         "per_layer": st["per_layer"]}
        # the bytes the stage's kernels really move (committed counter
        # summary of the same sources and tile), at this run's stage time:
        # scratch round trips and re-reads count here, not in GB_s
        tb = measured_traffic(name, sname, tile) if len(plans) == 1 and not split else None
        if tb is not None:
            tgbs = tb * st["launches"] / sec / 1e9
            detail[sname]["traffic_GB_s"] = round(tgbs, 1)
            detail[sname]["traffic_hbm_frac"] = round(tgbs / PEAK_HBM_GBS, 4)

    # dominant kernel: largest time share of the step
    dom = max(stages, key=lambda k: stages[k]["ms_total"])
    st = stages[dom]
    avg_s = st["ms_total"] * 1e-3 / st["launches"]
    ai = flop_x * st["flop"] / st["bytes"] if st["bytes"] else 0.0
    ridge = peak_mm * 1e12 / (PEAK_HBM_GBS * 1e9)
    if dom == "contraction" and ai > ridge:
        ach = flop_x * st["flop"] / st["launches"] / avg_s / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": peak_mm,
                "unit": "TFLOP/s", "frac": round(ach / peak_mm, 4)}
    else:
        ach = st["bytes"] / st["launches"] / avg_s / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4)}
    roof["kernel"] = dom
    roof["avg_launch_us"] = round(avg_s * 1e6, 2)
    traffic = measured_traffic(name, dom, tile) if len(plans) == 1 and not split else None
    roof["traffic"] = traffic
    roof["traffic_source"] = (f"profiles/traffic_{name}_{tile}.json: rocprofv3 FETCH_SIZE and "
                              f"WRITE_SIZE of this kernel source, scaled by a device copy"
                              if traffic is not None else None)

    L0 = wl.layers[0]
    cfg = {"workload": name, "layers": len(wl.layers), "B": L0.B,
           "M": L0.M, "N": wl.layers[-1].N, "H": L0.H, "W": L0.W,
           "r": [L.r for L in wl.layers] if len(wl.layers) > 1 else L0.r,
           "pad": [L.pad for L in wl.layers] if len(wl.layers) > 1 else L0.pad,
           "base": [TILE_NAMES.get(p.info["tile"], "F(2x2,3x3)") for p in plans]
                   if tile != "f23" else "F(2x2,3x3)",
           "nesting_depth": [p.info["n"] for p in plans],
           "pipeline_parts": [p.info["pipeline_parts"] for p in plans],
           "launch": "hip-graph replay" if graph else "eager"}
    return {"plans": plans, "ms_step": ms_step, "ms_step_eager": ms_step_eager,
            "value": direct_flop / (ms_step * 1e-3) / 1e12, "direct_flop": direct_flop,
            "stages": detail, "roofline": roof, "config": cfg, "kx_ms": kx_ms,
            "kx_bytes": kx_bytes,
            "kx_first_ms": kx_first_ms, "split": split, "y": y_timed}


def kernel_transform_entry(ms: float, nbytes: float) -> dict:
    """The cached kernel transform, timed apart from the step: its algorithmic
    bytes (w + U) and their rate against the HBM peak."""
    gbs = nbytes / (ms * 1e-3) / 1e9 if ms > 0 else 0.0
    return {"ms_once": round(ms, 4), "bytes": nbytes, "GB_s": round(gbs, 1),
            "hbm_frac": round(gbs / PEAK_HBM_GBS, 4), "bound": "hbm"}


def close(res):
    for p in res["plans"]:
        p.close()
    res["plans"] = []


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c5_r31")
    ap.add_argument("--tile", choices=["f23", "f33", "auto", "ld", "mix"], default="auto",
                    help="Winograd base: F(2x2,3x3) nests (any r <= 31); F(3x3,3x3) nests for "
                         "the dense layers with r <= 9 (others keep F(2x2,3x3)); the "
                         "library's per-layer choice (NWG_TILE_AUTO); the linear "
                         "decomposition on F(2x2,3x3) (Sec. II.B) for the dense layers with "
                         "r > 1; or the mixed nest (F(2,3) at levels 1-2, F(3,3) above) for "
                         "the dense layers with r >= 8")
    ap.add_argument("--precision", choices=["fp32", "bf16_split"], default="fp32",
                    help="contraction arithmetic: fp32 MFMA, or the two-term bf16 split of U "
                         "and V on bf16 MFMA with fp32 accumulation (plans that can take it)")
    ap.add_argument("--graph", action="store_true",
                    help="time the step as replays of one HIP graph holding every layer's "
                         "launches (per-kernel times still come from an eager timed region)")
    ap.add_argument("--pipeline-parts", type=int, default=0,
                    help="input-transform/contraction pieces on two streams (0: the library's "
                         "default for each plan, 1: off)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="approximate CPU time for the oracle baseline sample (and parity)")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle: no cpu_baseline and no parity fields")
    ap.add_argument("--no-compare", action="store_true",
                    help="skip the all-F(2x2,3x3) comparison step (e.g. under a counter run)")
    ap.add_argument("--no-per-config", action="store_true",
                    help="skip the other workloads' lines (per_config)")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="first copy a float32 buffer of this many MiB (a plain copy kernel of "
                         "known size, to scale hardware byte counters)")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="no GPU work: turn two rocprofv3 --pmc counter files (FETCH_SIZE, "
                         "WRITE_SIZE) of a --calibrate-copy-mib run into "
                         "profiles/traffic_<workload>_<tile>.json")
    args = ap.parse_args()
    if args.traffic_from:
        res = traffic_from_counters(args.workload, args.tile, args.traffic_from[0],
                                    args.traffic_from[1], args.calibrate_copy_mib or 1024)
        print(json.dumps(res, indent=1))
        return
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU only (got --gpus {args.gpus}); the path "
              f"would shard over output tiles or Winograd points, which the library does not do.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2102_13272_amd import nwg
    from paper_2102_13272_amd.workloads import WORKLOADS

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    nwg.load_library()
    torch.cuda.set_device(0)
    if args.calibrate_copy_mib > 0:
        n = args.calibrate_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    res = run_workload(torch, nwg, args.workload, args.tile, args.precision, args.steps,
                       args.warmup, args.pipeline_parts, args.graph)
    cfg = res["config"]
    out = {
        "metric": METRIC, "value": round(res["value"], 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(res["ms_step"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16-split/f32-acc" if res["split"] else "f32",
        "data": "synthetic", "config": cfg, "roofline": res["roofline"],
        "stages": res["stages"],
        "kernel_transform_ms_once": round(res["kx_ms"], 4),
        "kernel_transform": kernel_transform_entry(res["kx_ms"], res["kx_bytes"]),
        "kernel_transform_ms_first_call": round(res["kx_first_ms"], 4),
        "value_incl_kernel_transform": round(
            res["direct_flop"] / ((res["ms_step"] + res["kx_ms"]) * 1e-3) / 1e12, 3),
        "direct_flop_per_step": res["direct_flop"],
    }
    if args.graph:
        out["ms_per_step_eager"] = round(res["ms_step_eager"], 4)
    y_main = res["y"]
    compare_tile = any(p.info["tile"] != nwg.NWG_TILE_F2X2_3X3 for p in res["plans"])
    close(res)
    y_f23 = None
    if not args.no_compare and compare_tile:
        # the same workload with every layer on F(2x2,3x3) nests, timed the
        # same way in the same run, for comparison
        r2 = run_workload(torch, nwg, args.workload, "f23", args.precision, args.steps,
                          args.warmup)
        out["f2x2_3x3_only"] = {
            "ms_per_step": round(r2["ms_step"], 4), "value": round(r2["value"], 3),
            "roofline": {k: r2["roofline"][k] for k in ("bound", "frac", "kernel")},
            "stages": {k: {f: v[f] for f in ("ms_per_step", "GB_s", "hbm_frac", "TFLOP_s",
                                              "mfma_frac", "traffic_GB_s", "traffic_hbm_frac")
                           if f in v}
                       for k, v in r2["stages"].items()},
            "kernel_transform": kernel_transform_entry(r2["kx_ms"], r2["kx_bytes"])}
        y_f23 = r2["y"]
        close(r2)
    failed = []
    if not args.no_cpu_baseline:
        outs = {"timed": y_main}
        if y_f23 is not None:
            outs["f2x2_3x3_only"] = y_f23
        base, par = cpu_baseline(args.workload, args.cpu_seconds, outs)
        out["cpu_baseline"] = base
        out["parity"] = par["timed"]
        if "f2x2_3x3_only" in par:
            out["f2x2_3x3_only"]["parity"] = par["f2x2_3x3_only"]
        failed += [args.workload + ("" if k == "timed" else f" ({k})")
                   for k, v in par.items() if not v["ok"]]
    if not args.no_per_config and args.workload == "c5_r31":
        # the other configs of the benchmark, each timed the same way, with its
        # dominant kernel's roofline and (unless skipped) its parity
        per = {}
        for name in ("c1_r4_valid", "c2_r7", "c3_r13", "c4_sr_stack"):
            rk = run_workload(torch, nwg, name, args.tile, args.precision, args.steps,
                              args.warmup)
            ent = {"ms_per_step": round(rk["ms_step"], 4), "value": round(rk["value"], 3),
                   "unit": "TFLOP/s", "config": rk["config"],
                   "roofline": {k: rk["roofline"][k]
                                for k in ("bound", "achieved", "peak", "unit", "frac",
                                          "kernel", "avg_launch_us", "traffic",
                                          "traffic_source")},
                   "stages": {k: {f: v[f] for f in ("ms_per_step", "GB_s", "hbm_frac",
                                                     "TFLOP_s", "mfma_frac", "traffic_GB_s",
                                                     "traffic_hbm_frac") if f in v}
                              for k, v in rk["stages"].items()},
                   "kernel_transform": kernel_transform_entry(rk["kx_ms"], rk["kx_bytes"])}
            y_k = rk["y"]
            close(rk)
            if not args.no_cpu_baseline:
                bk, pk = cpu_baseline(name, 2.0, {"timed": y_k})
                ent["cpu_baseline"] = bk
                ent["parity"] = pk["timed"]
                if not pk["timed"]["ok"]:
                    failed.append(name)
            per[name] = ent
        out["per_config"] = per
    print(json.dumps(out), flush=True)
    if failed:
        print(f"bench.py: output outside the fp32 bar against the oracle: {failed}",
              file=sys.stderr)
        sys.exit(3)


if __name__ == "__main__":
    main()
