"""Pins for the oracle's block composition, ``oracle.block``: the paper's
network block pattern (the basic blocks of its PyTorch comparison, Table 2)
as convolution (Algorithm 1) -> multivector activation (Algorithm 3) ->
convolution -> activation, kept in fp64 end to end.

Each pin is chosen so that a plausible mistake in the composition fails it:
  * an explicit chain of the oracle's pinned single layers, compared bit for
    bit with a different activation per layer (catches a swapped
    activation/convolution order, a dropped or repeated layer, the wrong
    activation on a layer, an fp32-rounded intermediate);
  * a closed form: a unit scalar centre tap in both layers, zero conv bias
    and a Linear gate with zero weight and bias (sigma(0) = 1/2 in both
    activations) returns the input cropped by d_filter - 1 on each side,
    divided by 4, bit for bit (a dropped activation gives /2, an extra one /8,
    a wrong crop shifts the window);
  * scalar-only filters: the block is then a real convolution per blade with
    the activation's gate mixing the blades, computed here independently with
    torch's fp64 convolution and sigmoid;
  * translation equivariance (no padding): the block of a cropped input is
    the same window of the block's full output, bit for bit; the full-size
    GPU tests of the blocks rely on it.
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import AGG_LINEAR, AGG_MEAN, AGG_SUM, random_conv_case


def _layers(seed, k, C_in, C_mid, C_out, d_f, acts):
    rng = np.random.default_rng(seed)
    nb = 1 << k
    out = []
    for (ci, co), a in zip(((C_in, C_mid), (C_mid, C_out)), acts):
        bound = 1.0 / np.sqrt(ci * d_f ** k)
        f = rng.uniform(-bound, bound, (ci, co) + (d_f,) * k + (nb,)).astype(np.float32)
        b = (0.1 * rng.standard_normal((co, nb))).astype(np.float32)
        act = None
        if a is not None:
            mode, blades = a
            aw = ab = None
            if mode == AGG_LINEAR:
                aw = rng.standard_normal((co, len(blades))).astype(np.float32)
                ab = (0.1 * rng.standard_normal(co)).astype(np.float32)
            act = (mode, blades, aw, ab)
        out.append((f, b, act))
    return out


CHAIN_CASES = [
    # k, g, B, C_in, C_mid, C_out, d_image, d_filter, activations of the two layers
    (2, (1, -1), 2, 3, 5, 4, 11, 3, [(AGG_LINEAR, (0, 1, 2, 3)), (AGG_MEAN, (1, 3))]),
    (2, (1, 1), 1, 2, 3, 2, 9, 2, [(AGG_SUM, (0, 2)), (AGG_LINEAR, (3,))]),
    (3, (1, 1, 1), 2, 2, 3, 2, 8, 3,
     [(AGG_MEAN, tuple(range(8))), (AGG_LINEAR, (0, 4, 7))]),
    (1, (-1,), 3, 4, 3, 5, 20, 4, [(AGG_LINEAR, (0, 1)), (AGG_SUM, (1,))]),
    (2, (0, -1), 2, 2, 2, 3, 8, 3, [None, (AGG_MEAN, (0, 1, 2, 3))]),
]


@pytest.mark.parametrize("case", CHAIN_CASES, ids=lambda c: "k%d_g%s" % (c[0], c[1]))
def test_block_is_the_explicit_chain(case):
    k, g, B, C_in, C_mid, C_out, d_image, d_f, acts = case
    rng = np.random.default_rng(31 + k)
    x = rng.standard_normal((B, C_in) + (d_image,) * k + (1 << k,)).astype(np.float32)
    layers = _layers(7 * k + d_f, k, C_in, C_mid, C_out, d_f, acts)
    y = oracle.block(x, layers, g)
    # the same chain spelt out with the single-layer oracle functions
    (f1, b1, a1), (f2, b2, a2) = layers
    h = oracle.conv_nd(x, f1, b1, g)
    if a1 is not None:
        h = oracle.act(h, *a1)
    r = oracle.conv_nd(h, f2, b2, g)
    r = oracle.act(r, *a2)
    d_out = d_image - 2 * (d_f - 1)
    assert y.dtype == np.float64
    assert y.shape == (B, C_out) + (d_out,) * k + (1 << k,)
    assert np.array_equal(y, r)
    # the order matters: activation before the first convolution, or the
    # last activation left out, give a different result
    if a1 is not None and a1[0] != AGG_LINEAR:  # (a Linear gate is sized for C_mid)
        swapped = oracle.act(oracle.conv_nd(oracle.conv_nd(oracle.act(x, *a1), f1, b1, g),
                                            f2, b2, g), *a2)
        assert not np.allclose(y, swapped, rtol=1e-6, atol=1e-9)
    assert not np.allclose(y, oracle.conv_nd(h, f2, b2, g), rtol=1e-6, atol=1e-9)


@pytest.mark.parametrize("k,g,d_f", [(1, (-1,), 3), (2, (1, 1), 3), (2, (1, -1), 5),
                                     (3, (1, 1, 1), 3), (3, (-1, 0, 1), 1)])
def test_unit_centre_tap_zero_gate_block_is_quarter_crop(k, g, d_f):
    nb = 1 << k
    C, B, d_image = 3, 2, 4 * d_f + 3
    rng = np.random.default_rng(5 + k)
    x = rng.standard_normal((B, C) + (d_image,) * k + (nb,)).astype(np.float32)
    f = np.zeros((C, C) + (d_f,) * k + (nb,), np.float32)
    centre = (d_f // 2,) * k
    for c in range(C):
        f[(c, c) + centre + (0,)] = 1.0
    zero_b = np.zeros((C, nb), np.float32)
    gate = (AGG_LINEAR, tuple(range(nb)), np.zeros((C, nb), np.float32),
            np.zeros(C, np.float32))
    y = oracle.block(x, [(f, zero_b, gate), (f, zero_b, gate)], g)
    h = d_f - 1  # d_filter - 1 over two layers: (d_f - 1) / 2 per side each
    crop = (slice(None), slice(None)) + (slice(h, d_image - h),) * k
    assert np.array_equal(y, x[crop].astype(np.float64) / 4.0)


def _torch_act(y, mode, blades, aw, ab):
    """Algorithm 3 written with torch ops on [B, C, spatial..., N_B], fp64:
    one gate per multivector from the selected blades, sigmoid, scale all
    blades."""
    sel = y[..., list(blades)]
    C = y.shape[1]
    shape = (1, C) + (1,) * (y.dim() - 3) + (len(blades),)
    if mode == AGG_LINEAR:
        s = (sel * torch.from_numpy(aw.astype(np.float64)).reshape(shape)).sum(-1)
        s = s + torch.from_numpy(ab.astype(np.float64)).reshape(shape[:-1])
    elif mode == AGG_SUM:
        s = sel.sum(-1)
    else:
        s = sel.mean(-1)
    return y * torch.sigmoid(s).unsqueeze(-1)


def _torch_scalar_conv(y, f, b, k):
    """Convolution with scalar-only filters: a real convolution of every blade
    plane with the filters' scalar parts (cross-correlation, no padding),
    plus the bias."""
    conv = {1: torch.nn.functional.conv1d, 2: torch.nn.functional.conv2d,
            3: torch.nn.functional.conv3d}[k]
    nb = y.shape[-1]
    w = torch.from_numpy(np.moveaxis(f[..., 0].astype(np.float64), 0, 1).copy())  # [co, ci, taps]
    planes = [conv(y[..., j], w) for j in range(nb)]
    out = torch.stack(planes, dim=-1)
    bt = torch.from_numpy(b.astype(np.float64)).reshape((1, b.shape[0]) + (1,) * k + (nb,))
    return out + bt


@pytest.mark.parametrize("k,g", [(2, (1, -1)), (3, (1, 1, 1)), (2, (-1, -1)), (1, (1,))])
def test_scalar_filter_block_is_per_blade_real_conv(k, g):
    nb = 1 << k
    B, C_in, C_mid, C_out, d_f = 2, 3, 4, 2, 3
    d_image = 9 if k < 3 else 7
    rng = np.random.default_rng(40 + k)
    x = rng.standard_normal((B, C_in) + (d_image,) * k + (nb,)).astype(np.float32)
    acts = [(AGG_LINEAR, tuple(range(nb))), (AGG_MEAN, tuple(range(0, nb, 2)))]
    layers = _layers(50 + k, k, C_in, C_mid, C_out, d_f, acts)
    layers = [(np.where(np.arange(nb) == 0, f, 0).astype(np.float32), b, a)
              for f, b, a in layers]
    y = oracle.block(x, layers, g)
    t = torch.from_numpy(x.astype(np.float64))
    for f, b, a in layers:
        t = _torch_act(_torch_scalar_conv(t, f, b, k), *a)
    np.testing.assert_allclose(y, t.numpy(), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("k,g", [(2, (1, -1)), (3, (1, 1, 1))])
def test_block_translation_equivariance(k, g):
    nb = 1 << k
    B, C, d_f = 2, 3, 3
    d_image = 12 if k == 2 else 9
    rng = np.random.default_rng(60 + k)
    x = rng.standard_normal((B, C) + (d_image,) * k + (nb,)).astype(np.float32)
    layers = _layers(61 + k, k, C, C, C, d_f,
                     [(AGG_LINEAR, tuple(range(nb))), (AGG_MEAN, tuple(range(nb)))])
    y = oracle.block(x, layers, g)
    halo, ps = 2 * (d_f - 1), 3
    for org in [(0,) * k, (1,) * k, tuple(range(k))]:
        crop = (slice(1, 2), slice(None)) + tuple(slice(o, o + ps + halo) for o in org)
        win = (slice(1, 2), slice(None)) + tuple(slice(o, o + ps) for o in org)
        assert np.array_equal(oracle.block(x[crop], layers, g), y[win])


def test_block_crops_stack_as_a_batch():
    # the sampled check of the 3D block evaluates many crops at once as one
    # batch: batch entries are independent, so each row equals its crop alone
    k, g, nb, d_f = 3, (1, 1, 1), 8, 3
    _, x, _, _ = random_conv_case(3, k, g, 2, 2, 2, 8, d_f)
    layers = _layers(70, k, 2, 3, 2, d_f, [(AGG_MEAN, tuple(range(nb))), (AGG_SUM, (0, 7))])
    crops = [x[b:b + 1, :, z:z + 5, y:y + 5, w:w + 5] for b, z, y, w in
             [(0, 0, 0, 0), (1, 3, 1, 2), (0, 2, 3, 3)]]
    many = oracle.block(np.concatenate(crops), layers, g)
    for i, c in enumerate(crops):
        assert np.array_equal(many[i:i + 1], oracle.block(c, layers, g))
