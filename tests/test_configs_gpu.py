"""Full-size parity on the benchmark workloads, run through the C ABI in
the launch configuration the benchmark times (clifford_conv_nd, automatic
kernel choice, activation fused into the convolution for the blocks).

Every workload is compared with the fp64 oracle in full except the 3D block
(8.2 TFLOP, several minutes of oracle time), which is checked on
  * batch entry 0 in full (the oracle's block on that slice), and
  * >= 10^5 seeded random (b, c_out, p) outputs across all of B: random
    (b, p) with every output channel.  The oracle evaluates them as one batch
    of crops: with no padding the block of the input window that an output
    reads (d_filter - 1 halo per layer and side) equals that output of the
    full block (translation equivariance, pinned on the CPU), and batch
    entries are independent.
Gate: normwise relative error <= 1e-4; the element-wise relative error over
|r| >= 1e-3 max|r| is printed beside it (see gpu_util).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2507_01040_amd as P
import workloads as W
from gpu_util import assert_parity_report, dev

pytestmark = pytest.mark.gpu


def _gpu_block(w: W.Workload, x, params):
    """The benchmark's pass: every layer through clifford_conv_nd with the
    bias and (if any) activation fused."""
    xt = dev(x)
    ts = []
    for li, (shape, act) in enumerate(zip(w.layers, w.acts)):
        p = params[li]
        a = None
        if act is not None:
            a = (act.mode, act.blades,
                 dev(p.act_weight) if p.act_weight is not None else None,
                 dev(p.act_bias) if p.act_bias is not None else None)
        ts.append((dev(p.filters), dev(p.bias), a))
    y = P.block_forward(xt, ts, w.layers[0].g)
    torch.cuda.synchronize()
    out = y.cpu().numpy()
    del xt, ts, y
    torch.cuda.empty_cache()
    return out


def _oracle_layers(w: W.Workload, params):
    return [(p.filters, p.bias,
             None if a is None else (a.mode, a.blades, p.act_weight, p.act_bias))
            for p, a in zip(params, w.acts)]


def test_c1_full():
    w = W.WORKLOADS["conv2d_c4_d16"]
    x, ps = W.make_inputs(w)
    y = _gpu_block(w, x, ps)
    ref = oracle.conv_nd(x, ps[0].filters, ps[0].bias, w.layers[0].g)
    assert_parity_report(y, ref, what="conv2d_c4_d16 (full)")


def test_small_block_full():
    # the small-block workload through the block entry point (one fused
    # launch), every output against the oracle's fp64 block
    w = W.WORKLOADS["block2d_c4_d18"]
    x, ps = W.make_inputs(w)
    layers = []
    for p, act in zip(ps, w.acts):
        layers.append((dev(p.filters), dev(p.bias),
                       (act.mode, act.blades, dev(p.act_weight), dev(p.act_bias))))
    y = P.block2(dev(x), layers[0], layers[1], w.layers[0].g)
    torch.cuda.synchronize()
    ref = oracle.block(x, _oracle_layers(w, ps), w.layers[0].g)
    assert_parity_report(y.cpu().numpy(), ref, what="block2d_c4_d18 (full)")


# the fp64 oracle takes up to about a minute on these (all host cores)
HEAVY = pytest.mark.timeout(600)


@HEAVY
@pytest.mark.parametrize("name", ["conv2d_c64_d128", "conv3d_c32_d32", "conv1d_c64_d60"])
def test_single_conv_full(name):
    w = W.WORKLOADS[name]
    x, ps = W.make_inputs(w)
    y = _gpu_block(w, x, ps)
    ref = oracle.conv_nd(x, ps[0].filters, ps[0].bias, w.layers[0].g)
    assert_parity_report(y, ref, what="%s (full)" % name)


@HEAVY
def test_block2d_full():
    w = W.WORKLOADS["block2d_c64_d130"]
    x, ps = W.make_inputs(w)
    y = _gpu_block(w, x, ps)
    ref = oracle.block(x, _oracle_layers(w, ps), w.layers[0].g)
    assert_parity_report(y, ref, what="block2d_c64_d130 (full)")


@pytest.fixture(scope="module")
def block3d():
    w = W.WORKLOADS["block3d_c64_d36"]
    x, ps = W.make_inputs(w)
    y = _gpu_block(w, x, ps)
    return w, x, ps, y


@HEAVY
def test_block3d_batch0_full(block3d):
    w, x, ps, y = block3d
    ref = oracle.block(x[0:1], _oracle_layers(w, ps), w.layers[0].g)
    assert_parity_report(y[0:1], ref, what="block3d_c64_d36 (batch entry 0 in full)")


@HEAVY
def test_block3d_random_samples(block3d):
    w, x, ps, y = block3d
    k, C_out = w.layers[0].k, w.layers[-1].C_out
    halo = sum(l.d_filter - 1 for l in w.layers)
    d_final = w.layers[-1].d_out
    n_pos = (100_000 + C_out - 1) // C_out  # (b, p) pairs, every c_out each
    rng = np.random.default_rng(2024)
    bs = rng.integers(0, w.layers[0].B, n_pos)
    org = rng.integers(0, d_final, (n_pos, k))
    crops = np.stack([x[b][(slice(None),) + tuple(slice(o, o + halo + 1) for o in org[i])]
                      for i, b in enumerate(bs)])
    ref = oracle.block(crops, _oracle_layers(w, ps), w.layers[0].g)
    ref = ref.reshape(n_pos, C_out, -1)
    got = np.stack([y[b][(slice(None),) + tuple(org[i])] for i, b in enumerate(bs)])
    assert got.shape == ref.shape
    assert len(set(bs.tolist())) == w.layers[0].B
    assert_parity_report(got, ref, what="block3d_c64_d36 (%d random (b, c_out, p) outputs)"
                         % (n_pos * C_out))
