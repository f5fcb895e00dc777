"""Seeded synthetic inputs for the Clifford convolution workloads.

This module is shared by the tests, the benchmark and the smoke check. It
draws random numbers and describes shapes; it holds none of the layer's
arithmetic (no products, sums or activations), so both the CPU oracle and the
GPU path can be fed from it without sharing any of the method.

Layouts (blade index last, as in the paper's input/output protocol of the
"Optimization Performed" section, with the filters and bias written
blade-last as the typed arrays of Algorithm 1):
    input   [B, C_in,  d_image^k, N_B]
    filters [C_in, C_out, d_filter^k, N_B]
    bias    [C_out, N_B]
    output  [B, C_out, d_out^k, N_B],  d_out = d_image - d_filter + 1

Every array is float32, drawn with numpy's PCG64 generator seeded with
``1000 + index`` for the named workloads, in this fixed draw order:
input, filters1, bias1, actW1, actB1, filters2, bias2, actW2, actB2
(entries a workload does not use are not drawn).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence, Tuple

import numpy as np

AGG_LINEAR, AGG_SUM, AGG_MEAN = 0, 1, 2
AGG_NAMES = {AGG_LINEAR: "linear", AGG_SUM: "sum", AGG_MEAN: "mean"}


def n_blades(k: int) -> int:
    return 1 << k


@dataclasses.dataclass(frozen=True)
class ConvShape:
    k: int
    g: Tuple[int, ...]
    B: int
    C_in: int
    C_out: int
    d_image: int
    d_filter: int

    @property
    def nb(self) -> int:
        return n_blades(self.k)

    @property
    def d_out(self) -> int:
        return self.d_image - self.d_filter + 1

    def input_shape(self):
        return (self.B, self.C_in) + (self.d_image,) * self.k + (self.nb,)

    def filter_shape(self):
        return (self.C_in, self.C_out) + (self.d_filter,) * self.k + (self.nb,)

    def bias_shape(self):
        return (self.C_out, self.nb)

    def output_shape(self):
        return (self.B, self.C_out) + (self.d_out,) * self.k + (self.nb,)

    def useful_flops(self) -> int:
        """2 * B * C_out * C_in * N_B^2 * d_filter^k * d_out^k."""
        return (2 * self.B * self.C_out * self.C_in * self.nb * self.nb
                * self.d_filter ** self.k * self.d_out ** self.k)

    def algorithmic_bytes(self) -> int:
        """Input + filters + bias read once, output written once (fp32)."""
        n = 1
        for s in (self.input_shape(), self.filter_shape(), self.bias_shape(),
                  self.output_shape()):
            n += math.prod(s)
        return 4 * (n - 1)


@dataclasses.dataclass(frozen=True)
class ActSpec:
    mode: int
    blades: Tuple[int, ...]  # 0-based blade indices used for the gate


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    layers: Tuple[ConvShape, ...]
    acts: Tuple[Optional[ActSpec], ...]
    filter_bound: Tuple[float, ...]  # U(-a, a) half-width per layer
    bias_std: float
    act_bias_std: float = 0.1
    # "layers": one clifford_conv_nd launch per layer; "block2": the two-layer
    # block entry point (fused into one launch when small)
    entry: str = "layers"

    @property
    def useful_flops(self) -> int:
        return sum(l.useful_flops() for l in self.layers)


def _conv_layers(k, g, B, C, d_image, d_filter, n_layers):
    out = []
    d = d_image
    for _ in range(n_layers):
        out.append(ConvShape(k, tuple(g), B, C, C, d, d_filter))
        d = d - d_filter + 1
    return tuple(out)


def _fan_bound(C_in, d_filter, k):
    return 1.0 / math.sqrt(C_in * d_filter ** k)


# The workloads the benchmark and the full-size parity tests use.
WORKLOADS = {
    "conv2d_c4_d16": Workload(
        "conv2d_c4_d16", 1000,
        _conv_layers(2, (1, 1), 8, 4, 16, 3, 1), (None,),
        (_fan_bound(4, 3, 2),), bias_std=1.0),
    "conv2d_c64_d128": Workload(
        "conv2d_c64_d128", 1001,
        _conv_layers(2, (1, 1), 8, 64, 128, 3, 1), (None,),
        (_fan_bound(64, 3, 2),), bias_std=0.1),
    "conv3d_c32_d32": Workload(
        "conv3d_c32_d32", 1002,
        _conv_layers(3, (1, 1, 1), 8, 32, 32, 3, 1), (None,),
        (_fan_bound(32, 3, 3),), bias_std=0.1),
    "block2d_c64_d130": Workload(
        "block2d_c64_d130", 1003,
        _conv_layers(2, (1, -1), 8, 64, 130, 3, 2),
        (ActSpec(AGG_LINEAR, (0, 1, 2, 3)), ActSpec(AGG_LINEAR, (0, 1, 2, 3))),
        (_fan_bound(64, 3, 2),) * 2, bias_std=0.1),
    "block3d_c64_d36": Workload(
        "block3d_c64_d36", 1004,
        _conv_layers(3, (1, 1, 1), 8, 64, 36, 3, 2),
        (ActSpec(AGG_MEAN, tuple(range(8))), ActSpec(AGG_MEAN, tuple(range(8)))),
        (_fan_bound(64, 3, 3),) * 2, bias_std=0.1),
    # a block in the paper's small-parameter regime (C = 4, as the 2D tiny
    # workload): latency-bound, runs as one fused launch
    "block2d_c4_d18": Workload(
        "block2d_c4_d18", 1006,
        _conv_layers(2, (1, 1), 8, 4, 18, 3, 2),
        (ActSpec(AGG_LINEAR, (0, 1, 2, 3)), ActSpec(AGG_LINEAR, (0, 1, 2, 3))),
        (_fan_bound(4, 3, 2),) * 2, bias_std=1.0, entry="block2"),
    # the paper's 1-D layer (d_image 60, d_filter 17) at a GPU-sized batch
    "conv1d_c64_d60": Workload(
        "conv1d_c64_d60", 1005,
        _conv_layers(1, (-1,), 4096, 64, 60, 17, 1), (None,),
        (_fan_bound(64, 17, 1),), bias_std=0.1),
}
WORKLOAD_ORDER = list(WORKLOADS)


@dataclasses.dataclass
class LayerParams:
    filters: np.ndarray
    bias: np.ndarray
    act_weight: Optional[np.ndarray]  # [C_out, K] (Linear only)
    act_bias: Optional[np.ndarray]    # [C_out] (Linear only)


def _normal(rng, shape, std=1.0):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


def _uniform(rng, shape, a):
    return rng.uniform(-a, a, size=shape).astype(np.float32)


def make_inputs(w: Workload, batch_slice: Optional[slice] = None):
    """Returns (input, [LayerParams per layer]) as float32 numpy arrays."""
    rng = np.random.default_rng(w.seed)
    x = _normal(rng, w.layers[0].input_shape())
    params = []
    for li, (shape, act) in enumerate(zip(w.layers, w.acts)):
        f = _uniform(rng, shape.filter_shape(), w.filter_bound[li])
        b = _normal(rng, shape.bias_shape(), w.bias_std)
        aw = ab = None
        if act is not None and act.mode == AGG_LINEAR:
            aw = _normal(rng, (shape.C_out, len(act.blades)))
            ab = _normal(rng, (shape.C_out,), w.act_bias_std)
        params.append(LayerParams(f, b, aw, ab))
    if batch_slice is not None:
        x = np.ascontiguousarray(x[batch_slice])
    return x, params


def random_conv_case(seed: int, k: int, g: Sequence[int], B: int, C_in: int,
                     C_out: int, d_image: int, d_filter: int,
                     bias_std: float = 1.0):
    """Small seeded case for parity sweeps: input ~N(0,1), filters
    ~U(+-1/sqrt(C_in d_filter^k)), bias ~N(0, bias_std)."""
    s = ConvShape(k, tuple(g), B, C_in, C_out, d_image, d_filter)
    rng = np.random.default_rng(seed)
    x = _normal(rng, s.input_shape())
    f = _uniform(rng, s.filter_shape(), _fan_bound(C_in, d_filter, k))
    b = _normal(rng, s.bias_shape(), bias_std)
    return s, x, f, b


def random_act_case(seed: int, nb: int, B: int, C: int, P: int, mode: int,
                    K: int):
    """Seeded activation case: input [B, C, P, N_B] ~N(0,1), a random
    K-subset of blades, Linear weight ~N(0,1) and bias ~N(0,0.1)."""
    rng = np.random.default_rng(seed)
    x = _normal(rng, (B, C, P, nb))
    blades = tuple(int(v) for v in rng.permutation(nb)[:K])
    aw = _normal(rng, (C, K)) if mode == AGG_LINEAR else None
    ab = _normal(rng, (C,), 0.1) if mode == AGG_LINEAR else None
    return x, ActSpec(mode, blades), aw, ab


def batch_entry_normal(seed: int, b: int, entry_shape) -> np.ndarray:
    """N(0,1) float32 values of batch entry b of a large input, drawn from
    its own stream (seed, b), so any entry can be regenerated alone."""
    rng = np.random.default_rng([seed, b])
    return rng.standard_normal(size=tuple(entry_shape), dtype=np.float32)
