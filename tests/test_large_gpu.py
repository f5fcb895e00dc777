"""Maximum sizes: an input of more than 2^31 elements (8.6-8.7 GB) through the
convolution, the standalone activation and the streamed linear kernel, so
every 64-bit offset path is exercised.  Batch entries come from per-entry seeded streams
(workloads.batch_entry_normal), so the oracle regenerates only the entries
it checks; outputs are compared at sampled positions, including the last
batch entries, whose offsets exceed 2^31 elements."""
import numpy as np
import pytest
import torch

import oracle
import paper_2507_01040_amd as P
import workloads as W
from gpu_util import assert_parity, dev

pytestmark = pytest.mark.gpu

SEED = 4242


def test_conv_and_act_over_2_31_elements():
    s = W.ConvShape(2, (1, 1), 520, 64, 64, 128, 3)
    n_in = int(np.prod(s.input_shape()))
    assert n_in > 2 ** 31
    entry = s.input_shape()[1:]
    x = torch.empty(s.input_shape(), dtype=torch.float32, device="cuda:0")
    for b in range(s.B):
        x[b].copy_(torch.from_numpy(W.batch_entry_normal(SEED, b, entry)))
    _, _, f, bias = W.random_conv_case(SEED, 2, (1, 1), 1, 64, 64, 3, 3)
    y = P.conv_nd(x, dev(f), dev(bias), s.g)
    rng = np.random.default_rng(1)
    checks = [0, 255, 511, 512, 518, 519]
    for b in checks:
        xb = W.batch_entry_normal(SEED, b, entry)[None]
        cos = rng.integers(0, 64, 40)
        ps = np.concatenate([[0, s.d_out ** 2 - 1], rng.integers(0, s.d_out ** 2, 38)])
        ref = oracle.conv_points(xb, f, bias, s.g, np.zeros(40, np.int64), cos, ps)
        got = y[b].reshape(64, -1, 4)[torch.from_numpy(cos).cuda(),
                                       torch.from_numpy(ps).cuda()].cpu().numpy()
        assert_parity(got, ref, what="batch entry %d" % b)
    del y
    # standalone activation on the same 8.7 GB input, in place
    aw = rng.standard_normal((64, 4)).astype(np.float32)
    ab = rng.standard_normal(64).astype(np.float32)
    P.act_nd(x, P.AGG_LINEAR, (0, 1, 2, 3), dev(aw), dev(ab), out=x)
    for b in checks:
        xb = W.batch_entry_normal(SEED, b, entry)[None]
        ref = oracle.act(xb, P.AGG_LINEAR, (0, 1, 2, 3), aw, ab)[0]
        got = x[b].cpu().numpy()
        assert_parity(got, ref, what="act batch entry %d" % b)


def test_linear_over_2_31_elements():
    # the streamed linear kernel on an input of more than 2^31 elements
    # (2D, C = 32: 2^24 + 7 rows of 128 floats); the rows come in chunks of
    # 2^16, each from its own seeded stream, so the oracle regenerates only
    # the chunks it checks
    g, C, nb = (1, 1), 32, 4
    chunk = 1 << 16
    B = (1 << 24) + 7
    assert B * C * nb > 2 ** 31
    x = torch.empty((B, C, nb), dtype=torch.float32, device="cuda:0")
    n_chunks = (B + chunk - 1) // chunk

    def rows_of(c):
        n = min(chunk, B - c * chunk)
        return W.batch_entry_normal(SEED + 1, c, (n, C, nb))

    for c in range(n_chunks):
        x[c * chunk:c * chunk + chunk].copy_(torch.from_numpy(rows_of(c)))
    rng = np.random.default_rng(2)
    w = rng.uniform(-0.1, 0.1, (C, C, nb)).astype(np.float32)
    bias = rng.standard_normal((C, nb)).astype(np.float32)
    y = P.linear(x, dev(w), dev(bias), g)
    torch.cuda.synchronize()
    for c in (0, n_chunks // 2, n_chunks - 2, n_chunks - 1):
        xc = rows_of(c)
        sel = np.unique(np.concatenate([[0, len(xc) - 1], rng.integers(0, len(xc), 62)]))
        ref = oracle.linear(xc[sel], w, bias, g)
        got = y[torch.from_numpy(c * chunk + sel).cuda()].cpu().numpy()
        assert_parity(got, ref, what="rows of chunk %d" % c)
