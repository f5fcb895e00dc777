"""GPU parity on seeded random problems: k, signature (zero entries
included), batch, channel counts, filter and image sizes, the tile shape
(automatic or forced) and the fused activation (mode and blade subset) all
drawn at random, each output compared in full with the fp64 oracle (1e-4
normwise, as in the other parity tests).  The draw is fixed by its seed, so
the cases are the same on every run; their sizes keep the oracle to a
fraction of a second each."""
import itertools

import numpy as np
import pytest

import oracle
import paper_2507_01040_amd as P
from gpu_util import assert_parity, gpu_conv
from workloads import AGG_LINEAR, random_conv_case

pytestmark = pytest.mark.gpu

ALGOS = [P.ALGO_AUTO, P.ALGO_MFMA, P.ALGO_DIRECT, P.ALGO_MFMA_WIDE, P.ALGO_MFMA_MEDIUM,
         P.ALGO_MFMA_NARROW, P.ALGO_MFMA_TINY]
MAX_MACS = 1.5e8  # B C_in C_out N_B^2 d_filter^k d_out^k


def draw_cases(seed=20261202, n=128):
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        k = int(rng.integers(1, 4))
        g = tuple(int(v) for v in rng.integers(-1, 2, size=k))
        if not any(g):
            continue
        nb = 1 << k
        B = int(rng.integers(1, 5))
        C_in = int(rng.integers(1, 71))
        C_out = int(rng.integers(1, 71))
        df = int(rng.integers(1, 6 if k < 3 else 4))
        d = df + int(rng.integers(0, {1: 200, 2: 40, 3: 12}[k]))
        d_out = d - df + 1
        macs = B * C_in * C_out * nb * nb * df ** k * d_out ** k
        if macs > MAX_MACS:
            continue
        algo = ALGOS[int(rng.integers(len(ALGOS)))]
        act = None
        if rng.random() < 0.5:
            mode = int(rng.integers(0, 3))
            K = int(rng.integers(1, nb + 1))
            blades = tuple(sorted(int(b) for b in rng.choice(nb, size=K, replace=False)))
            act = (mode, blades)
        cases.append((k, g, B, C_in, C_out, d, df, algo, act, int(rng.integers(1 << 30))))
    return cases


CASES = draw_cases()


@pytest.mark.parametrize("case", CASES, ids=lambda c: "k%d-g%s-B%d-ci%d-co%d-d%d-f%d-a%d-%s" % (
    c[0], "".join({1: "+", -1: "-", 0: "0"}[v] for v in c[1]), c[2], c[3], c[4], c[5], c[6], c[7],
    "none" if c[8] is None else "m%d" % c[8][0]))
def test_random_problem(case):
    k, g, B, C_in, C_out, d, df, algo, act, seed = case
    _, x, f, b = random_conv_case(seed, k, g, B, C_in, C_out, d, df)
    act_args = None
    if act is not None:
        mode, blades = act
        rng = np.random.default_rng(seed + 1)
        aw = rng.standard_normal((C_out, len(blades))).astype(np.float32) if mode == AGG_LINEAR else None
        ab = rng.standard_normal(C_out).astype(np.float32) if mode == AGG_LINEAR else None
        act_args = (mode, blades, aw, ab)
    ref = oracle.conv_nd(x, f, b, g)
    if act_args is not None:
        ref = oracle.act(ref, *act_args)
    y = gpu_conv(g, x, f, b, act=act_args, algo=algo)
    assert_parity(y, ref, what=str(case))
