"""Call plans (paper_2507_01040_amd.conv_plan / block2_plan): the same
library call as conv_nd / block2 with the tensors checked and the arguments
marshalled once.  A plan's output equals the call's bit for bit, on the
stream it was made for and on another one, and a status other than CLIFF_OK
raises on the call that returns it."""
import numpy as np
import pytest
import torch

import oracle
import paper_2507_01040_amd as P
from gpu_util import assert_parity, dev
from workloads import random_conv_case

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("case", [(2, (1, 1), 3, 5, 6, 12, 3), (3, (1, -1, 0), 2, 4, 9, 8, 3),
                                  (1, (-1,), 5, 6, 7, 40, 17)], ids=str)
def test_conv_plan_matches_conv_nd(case):
    k, g, B, C_in, C_out, d, df = case
    _, x, f, b = random_conv_case(300, k, g, B, C_in, C_out, d, df)
    xt, ft, bt = dev(x), dev(f), dev(b)
    aw = torch.randn((C_out, 2), device="cuda:0")
    ab = torch.randn((C_out,), device="cuda:0")
    act = (P.AGG_LINEAR, (0, 1), aw, ab)
    ref = P.conv_nd(xt, ft, bt, g, act=act)
    plan = P.conv_plan(xt, ft, bt, g, act=act)
    for _ in range(3):
        y = plan()
    torch.cuda.synchronize()
    assert y is plan.out
    assert torch.equal(y, ref)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    plan.out.fill_(float("nan"))
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        plan(side)
    torch.cuda.synchronize()
    assert torch.equal(plan.out, ref)
    # and against the oracle
    r = oracle.act(oracle.conv_nd(x, f, b, g), act[0], act[1], aw.cpu().numpy().astype(np.float64),
                   ab.cpu().numpy().astype(np.float64))
    assert_parity(plan.out.cpu().numpy(), r, what=str(case))


def test_block2_plan_matches_block2():
    g = (1, -1)
    rng = np.random.default_rng(301)
    x = dev(rng.standard_normal((4, 3, 14, 14, 4)).astype(np.float32))
    f1 = dev((rng.uniform(-1, 1, (3, 5, 3, 3, 4)) / 6).astype(np.float32))
    f2 = dev((rng.uniform(-1, 1, (5, 2, 3, 3, 4)) / 8).astype(np.float32))
    b1 = dev(rng.standard_normal((5, 4)).astype(np.float32))
    b2 = dev(rng.standard_normal((2, 4)).astype(np.float32))
    l1 = (f1, b1, (P.AGG_MEAN, (0, 3), None, None))
    l2 = (f2, b2, (P.AGG_SUM, (1, 2), None, None))
    for path in (P.BLOCK_AUTO, P.BLOCK_TWO_LAUNCH, P.BLOCK_FUSED):
        ref = P.block2(x, l1, l2, g, path=path)
        plan = P.block2_plan(x, l1, l2, g, path=path)
        plan()
        plan()
        torch.cuda.synchronize()
        assert torch.equal(plan.out, ref), path


def test_plan_raises_on_a_failed_call():
    # the forced medium tile cannot stage this shape: the library returns
    # CLIFF_EUNSUPPORTED before launching anything, and the plan raises
    g = (1, 1)
    _, x, f, b = random_conv_case(302, 2, g, 2, 3, 5, 6, 6)
    plan = P.conv_plan(dev(x), dev(f), dev(b), g, algo=P.ALGO_MFMA_MEDIUM)
    with pytest.raises(P.CliffError) as e:
        plan()
    assert e.value.status == P.CLIFF_EUNSUPPORTED
