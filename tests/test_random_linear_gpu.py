"""GPU parity of the streamed linear-layer kernel on seeded random layers:
blade count, signature (zero entries included, which keep the sign
multiplies; the others take the negated weight copy where it fits), input
and output widths from {64, 128, 256} columns, batch (ragged last tiles, one
tile to several per wave), bias or none, and the fused activation, forced
with CLIFF_ALGO_MFMA_STREAM; every row compared with the fp64 oracle
(1e-4 normwise) and the NaN guard rows past B checked untouched.  The draw
is fixed by its seed."""
import numpy as np
import pytest

import oracle
from gpu_util import assert_parity
from test_linear_stream_gpu import _inputs, _run

pytestmark = pytest.mark.gpu


def draw_layers(seed=77, n=36):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        k = int(rng.integers(1, 4))
        nb = 1 << k
        g = tuple(int(v) for v in rng.integers(-1, 2, size=k))
        if not any(g):
            continue
        C_in = int(rng.choice([64, 128, 256])) // nb
        C_out = int(rng.choice([64, 128, 256])) // nb
        B = int(rng.choice([int(rng.integers(1, 200)), int(rng.integers(200, 40000))]))
        act = None
        if rng.random() < 0.5:
            K = int(rng.integers(1, nb + 1))
            act = (int(rng.integers(0, 3)),
                   tuple(sorted(int(b) for b in rng.choice(nb, size=K, replace=False))))
        out.append((g, C_in, C_out, B, bool(rng.random() < 0.8), act, int(rng.integers(1 << 20))))
    return out


LAYERS = draw_layers()


@pytest.mark.parametrize("case", LAYERS, ids=lambda c: "k%d-g%s-%dx%d-B%d" % (
    len(c[0]), "".join({1: "+", -1: "-", 0: "0"}[v] for v in c[0]), c[1], c[2], c[3]))
def test_random_linear(case):
    g, C_in, C_out, B, with_bias, act, seed = case
    nb = 1 << len(g)
    x, w, b = _inputs(seed, B, C_in, nb, C_out)
    if not with_bias:
        b = None
    host_act = None
    if act is not None:
        mode, blades = act
        rng = np.random.default_rng(seed + 1)
        aw = rng.standard_normal((C_out, len(blades))).astype(np.float32) if mode == 0 else None
        ab = rng.standard_normal(C_out).astype(np.float32) if mode == 0 else None
        host_act = (mode, blades, aw, ab)
    y, tail = _run(g, x, w, b, act=host_act, guard=40)
    ref = oracle.linear(x, w, b, g)
    if host_act is not None:
        ref = oracle.act(ref, *host_act)
    assert_parity(y, ref, what=str(case))
    assert np.isnan(tail).all(), "rows past B were written"
