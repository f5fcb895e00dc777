"""The library's launches captured in a HIP graph (through torch.cuda.graph):
replays must equal the eager results bit for bit (the kernels are
deterministic), with eager work and synchronisations between replays and
the inputs changed between replays.  The library records no memset or
allocation, only kernel launches on the caller's stream."""
import numpy as np
import pytest
import torch

import paper_2507_01040_amd as P
import workloads as W
from gpu_util import dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("k", [2, 3])
def test_graph_replay_matches_eager(k):
    g = (1, -1) if k == 2 else (1, 1, 1)
    nb = 1 << k
    s, x, f, b = W.random_conv_case(500 + k, k, g, 3, 8, 40, 14 if k == 2 else 9, 3)
    rng = np.random.default_rng(7)
    aw = rng.standard_normal((40, nb)).astype(np.float32)
    ab = rng.standard_normal(40).astype(np.float32)
    xt, ft, bt, awt, abt = dev(x), dev(f), dev(b), dev(aw), dev(ab)
    act = (P.AGG_LINEAR, tuple(range(nb)), awt, abt)
    out_g = torch.empty(s.output_shape(), device="cuda:0")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm up on the capture stream
        P.conv_nd(xt, ft, bt, g, act=act, out=out_g)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        P.conv_nd(xt, ft, bt, g, act=act, out=out_g)
    for rep in range(3):
        # new input values, eager reference, then a replay
        xt.copy_(dev(x * (1.0 + 0.25 * rep)))
        eager = P.conv_nd(xt, ft, bt, g, act=act)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_g, eager), "replay %d differs from eager" % rep


@pytest.mark.parametrize("path", [P.BLOCK_FUSED, P.BLOCK_TWO_LAUNCH], ids=["fused", "two_launch"])
def test_graph_replay_block2(path):
    # the two-layer block entry point, both paths, captured and replayed
    g = (1, 1)
    _, x, f1, b1 = W.random_conv_case(510, 2, g, 4, 4, 6, 18, 3)
    _, _, f2, b2 = W.random_conv_case(511, 2, g, 4, 6, 4, 16, 3)
    rng = np.random.default_rng(9)
    aw = dev(rng.standard_normal((6, 4)).astype(np.float32))
    ab = dev(rng.standard_normal(6).astype(np.float32))
    l1 = (dev(f1), dev(b1), (P.AGG_LINEAR, (0, 1, 2, 3), aw, ab))
    l2 = (dev(f2), dev(b2), (P.AGG_MEAN, (1, 2), None, None))
    xt = dev(x)
    ws = torch.empty((4, 6, 16, 16, 4), device="cuda:0")
    out_g = torch.empty((4, 4, 14, 14, 4), device="cuda:0")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        P.block2(xt, l1, l2, g, out=out_g, workspace=ws, path=path)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        P.block2(xt, l1, l2, g, out=out_g, workspace=ws, path=path)
    for rep in range(3):
        xt.copy_(dev(x * (1.0 - 0.3 * rep)))
        eager = P.block2(xt, l1, l2, g, path=path)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_g, eager), "replay %d differs from eager" % rep


def test_graph_replay_linear_stream():
    # the streamed linear kernel (persistent grid, buffer-descriptor stores)
    # captured and replayed, with its fused activation
    g = (1, 1)
    B, C = 40000, 32
    rng = np.random.default_rng(11)
    x = rng.standard_normal((B, C, 4)).astype(np.float32)
    xt = dev(x)
    wt = dev(rng.uniform(-0.1, 0.1, (C, C, 4)).astype(np.float32))
    bt = dev(rng.standard_normal((C, 4)).astype(np.float32))
    act = (P.AGG_SUM, (0, 3), None, None)
    out_g = torch.empty((B, C, 4), device="cuda:0")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        P.linear(xt, wt, bt, g, act=act, out=out_g)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        P.linear(xt, wt, bt, g, act=act, out=out_g)
    for rep in range(3):
        xt.copy_(dev(x * (1.0 - 0.3 * rep)))
        eager = P.linear(xt, wt, bt, g, act=act)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_g, eager), "replay %d differs from eager" % rep
