"""Seeded synthetic workloads for the nested-Winograd convolution.

This module only describes shapes and draws random inputs.  It contains none
of the method's arithmetic, so that the tests, the benchmark and the CPU
oracle can all take their inputs from it without sharing any computation.

Every array is drawn in float64 from numpy's PCG64 generator and cast to
float32 (the library computes in fp32).  Workload ``k`` (1-based) uses seed
``1000*k``; x is drawn first, then w.  In the super-resolution stack, layer
``i`` (1-based) draws its weight from seed ``4000+i``.

Weight scale: normal with variance 1/(M*r*r) (fan-in scaling), i.e. standard
deviation (M*r*r)**-0.5.

The shapes follow the problem statement of Sec. II.A (M input maps of HxW,
N groups of M-channel r x r kernels, N output maps, stride 1) and the kernel
sizes the paper targets (4x4 ... 31x31, Sec. I and V.A); the stack stands in
for the super-resolution networks of Table I / Sec. V.B with synthetic data.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np


@dataclass(frozen=True)
class Layer:
    """One stride-1 convolution: x[B][M][H][W] * w[N][M][r][r] -> y[B][N][Ho][Wo].

    depthwise: M == N channels, w[N][1][r][r], no sum over channels.
    """
    B: int
    M: int
    N: int
    H: int
    W: int
    r: int
    pad: int
    depthwise: bool = False

    @property
    def Ho(self) -> int:
        return self.H + 2 * self.pad - self.r + 1

    @property
    def Wo(self) -> int:
        return self.W + 2 * self.pad - self.r + 1

    @property
    def direct_flop(self) -> int:
        """FLOP of the direct convolution (one multiply + one add per tap)."""
        mk = 1 if self.depthwise else self.M
        return 2 * self.B * self.N * mk * self.Ho * self.Wo * self.r * self.r

    @property
    def w_shape(self):
        return (self.N, 1 if self.depthwise else self.M, self.r, self.r)


@dataclass(frozen=True)
class Workload:
    name: str
    layers: List[Layer]
    x_dist: str            # "uniform_pm1", "uniform_01" or "normal"
    w_dist: str            # "uniform_pm1" or "fanin_normal"
    seed: int
    layer_seeds: Optional[List[int]] = None   # per-layer weight seeds (stack only)
    note: str = field(default="")

    @property
    def direct_flop(self) -> int:
        return sum(L.direct_flop for L in self.layers)


def _same(r: int) -> int:
    return (r - 1) // 2


def _sr_stack() -> List[Layer]:
    B, H = 4, 256
    spec = [(1, 32, 5), (32, 5, 1), (5, 5, 3), (5, 5, 3), (5, 5, 3), (5, 5, 3),
            (5, 32, 1), (32, 1, 9)]
    return [Layer(B, m, n, H, H, r, _same(r)) for (m, n, r) in spec]


WORKLOADS = {
    "c1_r4_valid": Workload(
        "c1_r4_valid", [Layer(1, 4, 4, 16, 16, 4, 0)], "uniform_pm1", "uniform_pm1", 1000,
        note="4x4 kernel, 4->4 channels, 16x16, no padding (output 13x13)"),
    "c2_r7": Workload(
        "c2_r7", [Layer(1, 32, 32, 64, 64, 7, 3)], "uniform_pm1", "fanin_normal", 2000,
        note="7x7 kernel, 32->32 channels, 64x64, same padding"),
    "c3_r13": Workload(
        "c3_r13", [Layer(8, 64, 64, 56, 56, 13, 6)], "normal", "fanin_normal", 3000,
        note="13x13 kernel, B=8, 64->64 channels, 56x56, same padding"),
    "c4_sr_stack": Workload(
        "c4_sr_stack", _sr_stack(), "uniform_01", "fanin_normal", 4000,
        layer_seeds=[4000 + i for i in range(1, 9)],
        note="super-resolution-shaped stack of 8 convolutions on 4 images of 256x256"),
    "c5_r31": Workload(
        "c5_r31", [Layer(16, 128, 128, 56, 56, 31, 15)], "normal", "fanin_normal", 5000,
        note="31x31 large-kernel backbone layer, B=16, 128->128 channels, 56x56, same padding"),
    "dw7_pnasnet": Workload(
        "dw7_pnasnet", [Layer(8, 54, 54, 83, 83, 7, 3, depthwise=True)], "normal",
        "fanin_normal", 6000,
        note="depthwise 7x7 on 54 channels of 83x83 (the shape of Table I's depth-wise row), "
             "B=8, same padding"),
    "srcnn_955": Workload(
        "srcnn_955", [Layer(1, 1, 64, 256, 256, 9, 4), Layer(1, 64, 32, 256, 256, 5, 2),
                      Layer(1, 32, 1, 256, 256, 5, 2)], "uniform_01", "fanin_normal", 7000,
        layer_seeds=[7001, 7002, 7003],
        note="the three SRCNN layers of Table I as one chain, (Cout, Cin, H, W) = "
             "(64, 1, 256, 256), (32, 64, 256, 256), (1, 32, 256, 256), same padding"),
}

# Order in which the workloads are listed (1-based index k matches seed 1000*k).
ORDER = ["c1_r4_valid", "c2_r7", "c3_r13", "c4_sr_stack", "c5_r31", "dw7_pnasnet", "srcnn_955"]


def _draw(rng: np.random.Generator, shape, dist: str, fan_in: int = 1) -> np.ndarray:
    if dist == "uniform_pm1":
        a = rng.uniform(-1.0, 1.0, size=shape)
    elif dist == "uniform_01":
        a = rng.uniform(0.0, 1.0, size=shape)
    elif dist == "normal":
        a = rng.standard_normal(size=shape)
    elif dist == "fanin_normal":
        a = rng.standard_normal(size=shape) * (1.0 / np.sqrt(fan_in))
    elif dist == "small_int":
        a = rng.integers(-2, 3, size=shape).astype(np.float64)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return a.astype(np.float32)


def make_input(layer: Layer, dist: str, seed: int) -> np.ndarray:
    """x[B][M][H][W] as float32 from ``seed``."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return _draw(rng, (layer.B, layer.M, layer.H, layer.W), dist)


def make_weight(layer: Layer, dist: str, rng: np.random.Generator) -> np.ndarray:
    return _draw(rng, layer.w_shape, dist, fan_in=layer.w_shape[1] * layer.r * layer.r)


def make_workload(name: str):
    """Return (x, [w per layer]) for a named workload, float32, deterministic."""
    wl = WORKLOADS[name]
    first = wl.layers[0]
    rng = np.random.Generator(np.random.PCG64(wl.seed))
    x = _draw(rng, (first.B, first.M, first.H, first.W), wl.x_dist)
    if wl.layer_seeds is None:
        ws = [make_weight(first, wl.w_dist, rng)]
    else:
        ws = []
        for L, s in zip(wl.layers, wl.layer_seeds):
            ws.append(make_weight(L, wl.w_dist, np.random.Generator(np.random.PCG64(s))))
    return x, ws


def make_case(B, M, N, H, W, r, pad, seed, x_dist="uniform_pm1", w_dist="uniform_pm1",
              depthwise=False):
    """A single ad-hoc layer for tests: returns (Layer, x, w)."""
    L = Layer(B, M, N, H, W, r, pad, depthwise)
    rng = np.random.Generator(np.random.PCG64(seed))
    x = _draw(rng, (B, M, H, W), x_dist)
    w = _draw(rng, L.w_shape, w_dist, fan_in=L.w_shape[1] * r * r)
    return L, x, w
