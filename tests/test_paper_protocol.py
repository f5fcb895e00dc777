"""The paper's protocol puts the blade axis first for filters (N_B, C_in,
C_out, d_f^k) and bias (N_B, C_out) ("Optimization Performed", convolutional
layers); the library stores them blade-last.  from_paper_protocol converts:
checked element by element against the index map written out, and, through
the oracle, as the same layer."""
import itertools

import numpy as np
import pytest

import oracle
import paper_2507_01040_amd as P
from workloads import random_conv_case


@pytest.mark.parametrize("k", [1, 2, 3])
def test_index_map(k):
    nb = 1 << k
    rng = np.random.default_rng(k)
    C_in, C_out, df = 3, 2, 2
    fp = rng.standard_normal((nb, C_in, C_out) + (df,) * k).astype(np.float32)
    bp = rng.standard_normal((nb, C_out)).astype(np.float32)
    f, b = P.from_paper_protocol(fp, bp)
    assert f.shape == (C_in, C_out) + (df,) * k + (nb,) and f.flags["C_CONTIGUOUS"]
    assert b.shape == (C_out, nb)
    for j, ci, co in itertools.product(range(nb), range(C_in), range(C_out)):
        for q in itertools.product(range(df), repeat=k):
            assert f[(ci, co) + q + (j,)] == fp[(j, ci, co) + q]
    for j, co in itertools.product(range(nb), range(C_out)):
        assert b[co, j] == bp[j, co]
    assert P.from_paper_protocol(fp)[1] is None


def test_same_layer_through_the_oracle():
    g = (1, -1)
    _, x, f, b = random_conv_case(31, 2, g, 2, 3, 4, 7, 3)
    fp = np.ascontiguousarray(np.moveaxis(f, -1, 0))  # the paper's layout
    bp = np.ascontiguousarray(b.T)
    f2, b2 = P.from_paper_protocol(fp, bp)
    assert np.array_equal(oracle.conv_nd(x, f2, b2, g), oracle.conv_nd(x, f, b, g))


@pytest.mark.gpu
def test_gpu_layer_from_paper_layout():
    import torch
    from gpu_util import assert_parity, dev
    g = (-1, -1)
    _, x, f, b = random_conv_case(32, 2, g, 2, 5, 6, 12, 3)
    fp = dev(np.ascontiguousarray(np.moveaxis(f, -1, 0)))
    bp = dev(np.ascontiguousarray(b.T))
    ft, bt = P.from_paper_protocol(fp, bp)
    y = P.conv_nd(dev(x), ft, bt, g)
    torch.cuda.synchronize()
    assert_parity(y.cpu().numpy(), oracle.conv_nd(x, f, b, g))
