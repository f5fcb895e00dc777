"""GPU parity on 2D images of 2048 and more positions per row (Algorithm 1
sets no size limit).  Whole-row slabs do not fit in LDS there, so the
matrix-core kernel takes row-aligned blocks, whose slabs hold the d_filter
input rows of one output row segment; the host bounds checker walks the same
launches on the CPU (tests/test_host_bounds.py).

The inputs (up to 4.3 GB) are compared at sampled 8 x 8 output windows:
the four corners, windows straddling the 128-position row-segment
boundaries, the last columns, and random ones, every output channel.  The
oracle computes each window exactly from its input crop (no padding:
translation equivariance, pinned on the CPU)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2507_01040_amd as P
import workloads as W
from gpu_util import assert_parity_report, dev

pytestmark = pytest.mark.gpu

WIN = 8


def _windows(Do, seed):
    rng = np.random.default_rng(seed)
    last = Do - WIN
    org = [(0, 0), (0, last), (last, 0), (last, last), (Do // 2, 124), (Do // 3, 252),
           (7, last - 1)]
    org += [tuple(int(v) for v in rng.integers(0, last + 1, 2)) for _ in range(4)]
    return org


@pytest.mark.parametrize("B,C,d,algo", [
    (2, 16, 2050, P.ALGO_AUTO),
    (1, 64, 2050, P.ALGO_MFMA_WIDE),
    (1, 16, 4098, P.ALGO_AUTO),
    (1, 32, 3000, P.ALGO_MFMA_WIDE),   # rows of 2998 outputs: a partial last segment
], ids=["d2050-C16-auto", "d2050-C64-wide", "d4098-C16-auto", "d3000-C32-wide"])
def test_wide_image(B, C, d, algo):
    g = (1, 1)
    s = W.ConvShape(2, g, B, C, C, d, 3)
    rng = np.random.default_rng(d + C)
    x = W._normal(rng, s.input_shape())
    f = W._uniform(rng, s.filter_shape(), W._fan_bound(C, 3, 2))
    b = W._normal(rng, s.bias_shape(), 0.1)
    print("wide image B %d C %d d %d algo %d: %.1f GB input" % (B, C, d, algo, x.nbytes / 1e9),
          flush=True)
    xt = dev(x)
    y = torch.full(s.output_shape(), float("nan"), dtype=torch.float32, device="cuda:0")
    P.conv_nd(xt, dev(f), dev(b), g, out=y, algo=algo)
    torch.cuda.synchronize()
    del xt
    gots, refs = [], []
    for bb in range(B):
        for (oy, ox) in _windows(s.d_out, bb):
            crop = x[bb:bb + 1, :, oy:oy + WIN + 2, ox:ox + WIN + 2]
            refs.append(oracle.conv_nd(crop, f, b, g))
            gots.append(y[bb:bb + 1, :, oy:oy + WIN, ox:ox + WIN].cpu().numpy())
    # every output written (NaN-prefilled): a reduction on the GPU
    assert not torch.isnan(y).any().item()
    assert_parity_report(np.concatenate(gots), np.concatenate(refs),
                         what="2D d %d C %d B %d (%d windows)" % (d, C, B, len(refs)))
