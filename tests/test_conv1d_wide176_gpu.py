"""GPU parity of the 1-D matrix-core convolution's 176-position tile (4 x 1
waves of 2 x 11 MFMA tiles: 64 output channels x 176 flattened positions).
The quantisation model takes it for the paper's filter length (17) where its
blocks fill the last round of CUs better than the 128-position form's; the
host bounds checker walks the same launches (tests/test_host_bounds.py),
which also asserts that these shapes get it.

Outputs are compared with the fp64 oracle on runs of batch entries (entries
are independent, and the flattened blocks cross entry boundaries every 44
or 45 positions): the first and last 12 entries and 12 in the middle, every
output channel and position."""
import numpy as np
import pytest
import torch

import oracle
import paper_2507_01040_amd as P
import workloads as W
from gpu_util import assert_parity_report, dev

pytestmark = pytest.mark.gpu


def _entries(B):
    mid = B // 2 - 6
    return np.r_[0:12, mid:mid + 12, B - 12:B]


@pytest.mark.parametrize("B,C_in,C_out,d,algo,act", [
    (1024, 64, 64, 60, P.ALGO_AUTO, False),
    (1000, 64, 62, 60, P.ALGO_MFMA_WIDE, False),   # C_out below the tile's 64 channels
    (1001, 64, 64, 61, P.ALGO_AUTO, True),         # odd d_image: 4-byte input loads
    (2048, 128, 128, 60, P.ALGO_AUTO, True),       # two channel blocks
], ids=["B1024-C64", "B1000-C62-wide", "B1001-d61-act", "B2048-C128-act"])
def test_conv1d_176(B, C_in, C_out, d, algo, act):
    g = (-1,)
    df = 17
    rng = np.random.default_rng(B + C_out + d)
    x = W._normal(rng, (B, C_in, d, 2))
    f = W._uniform(rng, (C_in, C_out, df, 2), W._fan_bound(C_in, df, 1))
    b = W._normal(rng, (C_out, 2), 0.1)
    a_np = a_dev = None
    if act:
        aw = W._normal(rng, (C_out, 2), 0.5)
        ab = W._normal(rng, (C_out,), 0.1)
        a_np = (P.AGG_LINEAR, (0, 1), aw, ab)
        a_dev = (P.AGG_LINEAR, (0, 1), dev(aw), dev(ab))
    print("1-D B %d C %d->%d d %d algo %d act %s" % (B, C_in, C_out, d, algo, act), flush=True)
    y = torch.full((B, C_out, d - df + 1, 2), float("nan"), dtype=torch.float32, device="cuda:0")
    P.conv_nd(dev(x), dev(f), dev(b), g, act=a_dev, out=y, algo=algo)
    torch.cuda.synchronize()
    assert not torch.isnan(y).any().item()
    sel = _entries(B)
    ref = oracle.conv_nd(x[sel], f, b, g)
    if act:
        ref = oracle.act(ref, a_np[0], a_np[1], a_np[2], a_np[3])
    assert_parity_report(y.cpu().numpy()[sel], ref,
                         what="1-D 176-position tile B %d C %d->%d d %d" % (B, C_in, C_out, d))
