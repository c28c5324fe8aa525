"""Helpers for the GPU tests: run the HIP library through the C ABI on torch
device tensors, and compare against the CPU oracle with the fp32 bar.

Tolerance (fp32 path against the fp64 oracle): relative L2 error <= 1e-4
and max-abs error <= 1e-3 * max|y|.
"""
import numpy as np
import torch

from paper_2102_13272_amd import nwg

REL_L2 = 1e-4
MAX_ABS_FRAC = 1e-3


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")


def run_conv(x, w, pad, plan=None):
    B, M, H, W = x.shape
    N, _, r, _ = w.shape
    own = plan is None
    if own:
        plan = nwg.Plan(B, M, N, H, W, r, pad)
    xd, wd = dev(x), dev(w)
    y = torch.empty(plan.y_shape, dtype=torch.float32, device="cuda")
    plan.conv2d(xd, wd, y)
    torch.cuda.synchronize()
    out = y.cpu().numpy().astype(np.float64)
    if own:
        plan.close()
    return out


def errors(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    rel = np.linalg.norm(got - ref) / (den if den > 0 else 1.0)
    scale = np.abs(ref).max() if ref.size else 0.0
    mabs = np.abs(got - ref).max() if ref.size else 0.0
    return rel, mabs, scale


def assert_close(got, ref, rel_tol=REL_L2, abs_frac=MAX_ABS_FRAC, what=""):
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), what
    rel, mabs, scale = errors(got, ref)
    assert rel <= rel_tol, f"{what}: rel-L2 {rel:.3e} > {rel_tol}"
    assert mabs <= abs_frac * scale, f"{what}: max-abs {mabs:.3e} > {abs_frac} * {scale:.3e}"
    return rel, mabs
