"""GPU parity of the two-layer block entry point on seeded random small
blocks (the fused kernel's regime: k = 2, 3, up to 16 channels, small
images): signature (zero entries included), batch, the three channel counts,
filter and image sizes and both activations (mode and blade subset) drawn at
random; the fused path and the two-launch path each against the fp64
oracle's block, in full (1e-4 normwise).  The draw is fixed by its seed."""
import numpy as np
import pytest

import paper_2507_01040_amd as P
from gpu_util import assert_parity
from test_block_gpu import _case, _gpu, _ref

pytestmark = pytest.mark.gpu


def draw_blocks(seed=1202, n=40):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        k = int(rng.integers(2, 4))
        g = tuple(int(v) for v in rng.integers(-1, 2, size=k))
        if not any(g):
            continue
        nb = 1 << k
        df = int(rng.integers(1, 5 if k == 2 else 4))
        d = 2 * df - 1 + int(rng.integers(0, 24 if k == 2 else 8))
        C0, C1, C2 = (int(v) for v in rng.integers(1, 17, size=3))
        B = int(rng.integers(1, 5))
        acts = []
        for _ in range(2):
            if rng.random() < 0.3:
                acts.append(None)
                continue
            K = int(rng.integers(1, nb + 1))
            acts.append((int(rng.integers(0, 3)),
                         tuple(sorted(int(b) for b in rng.choice(nb, size=K, replace=False)))))
        # the fused kernel's LDS working set with one output slice per band:
        # both layers' input slices (with halos) and both layers' filters
        d1 = d - df + 1
        r1, r0 = df, 2 * df - 1
        lds = 4 * nb * (C0 * r0 * d ** (k - 1) + C1 * r1 * d1 ** (k - 1) +
                        (C0 * C1 + C1 * C2) * df ** k)
        if lds > 160 * 1024:
            continue
        out.append((g, B, C0, C1, C2, d, df, tuple(acts), int(rng.integers(1 << 20))))
    return out


BLOCKS = draw_blocks()


@pytest.mark.parametrize("path", [P.BLOCK_FUSED, P.BLOCK_TWO_LAUNCH], ids=["fused", "two_launch"])
@pytest.mark.parametrize("case", BLOCKS, ids=lambda c: "k%d-B%d-c%d.%d.%d-d%d-f%d" % (
    len(c[0]), c[1], c[2], c[3], c[4], c[5], c[6]))
def test_random_block(case, path):
    g, B, C0, C1, C2, d, df, acts, seed = case
    x, l1, l2 = _case(seed, g, B, C0, C1, C2, d, df, acts)
    assert_parity(_gpu(x, l1, l2, g, path), _ref(x, l1, l2, g), what=str(case))
