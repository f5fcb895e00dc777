"""clifford_block2_nd_noalloc: the block entry point for callers that cannot
allocate, whose two-launch path keeps the intermediate in the library's fixed
scratch array instead of a caller workspace.  Called through the C ABI, it
must give the same output as clifford_block2_nd with a workspace, bit for bit
(same kernels, same order) and within the 1e-4 normwise gate of the fp64
oracle, on two calls in a row where the second has the smaller input (the
array keeps the first call's contents), on a block small enough for the
fused path (no scratch), and must refuse an intermediate over the array's
size before enqueueing anything."""
import numpy as np
import pytest
import torch

import oracle
import paper_2507_01040_amd as P
import workloads as W
from gpu_util import assert_parity, dev

pytestmark = pytest.mark.gpu


def _block(seed, g, B, C_in, C_mid, C_out, d, df, acts):
    k = len(g)
    _, x, f1, b1 = W.random_conv_case(seed, k, g, B, C_in, C_mid, d, df, bias_std=0.1)
    _, _, f2, b2 = W.random_conv_case(seed + 1, k, g, 1, C_mid, C_out, d - df + 1, df,
                                      bias_std=0.1)
    rng = np.random.default_rng(seed + 2)
    layers = []
    for (f, b, a, c) in ((f1, b1, acts[0], C_mid), (f2, b2, acts[1], C_out)):
        act = None
        if a is not None:
            mode, blades = a
            aw = rng.standard_normal((c, len(blades))).astype(np.float32) \
                if mode == P.AGG_LINEAR else None
            ab = (0.1 * rng.standard_normal(c)).astype(np.float32) \
                if mode == P.AGG_LINEAR else None
            act = (mode, blades, aw, ab)
        layers.append((f, b, act))
    return x, layers


def _desc(act, keep):
    if act is None:
        return None
    mode, blades, aw, ab = act
    awt = dev(aw) if aw is not None else None
    abt = dev(ab) if ab is not None else None
    keep += [awt, abt]
    return P.make_act_desc(mode, blades, awt.data_ptr() if awt is not None else 0,
                           abt.data_ptr() if abt is not None else 0)


def _run(g, x, layers, noalloc):
    """The block through the C ABI: clifford_block2_nd_noalloc, or
    clifford_block2_nd with a torch-allocated workspace."""
    k = len(g)
    nb = 1 << k
    (f1, b1, a1), (f2, b2, a2) = layers
    B, C_in, d = x.shape[0], x.shape[1], x.shape[2]
    C_mid, C_out, df = f1.shape[1], f2.shape[1], f1.shape[2]
    d_mid, d_out = d - df + 1, d - 2 * df + 2
    keep = []
    xt, f1t, b1t, f2t, b2t = dev(x), dev(f1), dev(b1), dev(f2), dev(b2)
    d1, d2 = _desc(a1, keep), _desc(a2, keep)
    out = torch.full((B, C_out) + (d_out,) * k + (nb,), float("nan"), device="cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    if noalloc:
        st = P.clifford_block2_nd_noalloc(k, g, B, C_in, C_mid, C_out, d, df, xt.data_ptr(),
                                          f1t.data_ptr(), b1t.data_ptr(), d1, f2t.data_ptr(),
                                          b2t.data_ptr(), d2, out.data_ptr(), stream)
    else:
        ws = torch.empty((B, C_mid) + (d_mid,) * k + (nb,), device="cuda:0")
        keep.append(ws)
        st = P.clifford_block2_nd_path(k, g, B, C_in, C_mid, C_out, d, df, xt.data_ptr(),
                                       f1t.data_ptr(), b1t.data_ptr(), d1, f2t.data_ptr(),
                                       b2t.data_ptr(), d2, ws.data_ptr(), out.data_ptr(), stream,
                                       P.BLOCK_AUTO)
    torch.cuda.synchronize()
    return st, out.cpu().numpy()


LIN4, MEAN8 = (P.AGG_LINEAR, (0, 1, 2, 3)), (P.AGG_MEAN, tuple(range(8)))
# (g, B, C_in, C_mid, C_out, d_image, d_filter, acts); the first two run as
# two launches through the scratch (C > 16), the second smaller than the first
CALLS = [
    ((1, -1), 4, 24, 32, 20, 70, 3, (LIN4, (P.AGG_SUM, (1, 2)))),  # 1.2 M intermediate floats
    ((1, -1), 2, 20, 24, 24, 38, 3, (None, LIN4)),
    ((1, 1, 1), 2, 20, 18, 17, 14, 3, (MEAN8, MEAN8)),             # 3D, two launches
    ((1, 1), 3, 4, 4, 4, 18, 3, (LIN4, LIN4)),                     # fused: no scratch used
]


def test_noalloc_equals_block2_on_calls_in_a_row():
    for i, (g, B, C_in, C_mid, C_out, d, df, acts) in enumerate(CALLS):
        x, layers = _block(300 + i, g, B, C_in, C_mid, C_out, d, df, acts)
        st_ref, ref = _run(g, x, layers, noalloc=False)
        st, y = _run(g, x, layers, noalloc=True)
        assert st_ref == P.CLIFF_OK and st == P.CLIFF_OK, (i, P.STATUS_NAMES.get(st))
        assert np.array_equal(y, ref), "call %d differs from clifford_block2_nd" % i
        r = oracle.block(x, [(f, b, a) for f, b, a in layers], g)
        assert_parity(y, r, what="no-alloc call %d" % i)


def test_noalloc_refuses_an_intermediate_over_the_scratch():
    # B * C_mid * d_mid^2 * 4 = 1 * 64 * 258^2 * 4 = 17.0 M floats > 16 Mi
    g, B, C_in, C_mid, C_out, d, df = (1, 1), 1, 4, 64, 4, 260, 3
    assert B * C_mid * (d - df + 1) ** 2 * 4 > P.NOALLOC_SCRATCH_FLOATS
    x, layers = _block(400, g, B, C_in, C_mid, C_out, d, df, (None, None))
    st, y = _run(g, x, layers, noalloc=True)
    assert st == P.CLIFF_ESCRATCH, P.STATUS_NAMES.get(st)
    assert np.all(np.isnan(y))  # nothing was enqueued
