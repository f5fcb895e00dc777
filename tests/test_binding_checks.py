"""The Python binding checks every tensor before it calls the library.

The C ABI receives raw device pointers and cannot see the buffers behind
them, so a wrong shape, dtype or device must be caught in the binding: an
output buffer that is too small would be written out of bounds, and an
activation weight left on the host would be dereferenced by a kernel.  These
tests run on the CPU with "meta" tensors (shapes without storage): a wrong
shape must raise ValueError naming it, and a call whose shapes are all right
gets as far as the device check ("must be a GPU tensor").  The library itself
is replaced by a stub that fails the test if anything reaches it.
"""
import pytest
import torch

import paper_2507_01040_amd as P

AL, AS, AM = P.AGG_LINEAR, P.AGG_SUM, P.AGG_MEAN


def m(*shape):
    return torch.empty(shape, dtype=torch.float32, device="meta")


@pytest.fixture(autouse=True)
def no_library(monkeypatch):
    def fail(*a, **kw):
        raise AssertionError("the library was called")
    monkeypatch.setattr(P, "load", fail)


def _raises(fn, match):
    with pytest.raises(ValueError, match=match):
        fn()


# 2D: x [B=2, C_in=3, 9, 9, 4], filters [3, 5, 3, 3, 4], output [2, 5, 7, 7, 4]
X2, F2, B2 = (2, 3, 9, 9, 4), (3, 5, 3, 3, 4), (5, 4)
G2 = (1, 1)


def test_conv_nd_shapes():
    ok = dict(x=m(*X2), filters=m(*F2), bias=m(*B2), g=G2)
    _raises(lambda: P.conv_nd(**ok), "x must be a GPU tensor")
    _raises(lambda: P.conv_nd(**{**ok, "x": m(2, 3, 9, 9)}), "x has shape")
    _raises(lambda: P.conv_nd(**{**ok, "x": m(2, 3, 9, 8, 4)}), "x has shape")
    _raises(lambda: P.conv_nd(**{**ok, "x": m(2, 3, 9, 9, 8)}), "x has shape")
    _raises(lambda: P.conv_nd(**{**ok, "filters": m(4, 5, 3, 3, 4)}), "filters has shape")
    _raises(lambda: P.conv_nd(**{**ok, "filters": m(3, 5, 3, 2, 4)}), "filters has shape")
    _raises(lambda: P.conv_nd(**{**ok, "filters": m(3, 5, 11, 11, 4)}), "exceeds d_image")
    _raises(lambda: P.conv_nd(**{**ok, "bias": m(4, 4)}), "bias has shape")
    _raises(lambda: P.conv_nd(**{**ok, "bias": m(5, 2)}), "bias has shape")
    # the output: too small, too large, wrong layout
    _raises(lambda: P.conv_nd(**ok, out=m(2, 5, 7, 6, 4)), "out has shape")
    _raises(lambda: P.conv_nd(**ok, out=m(2 * 5 * 49 * 4)), "out has shape")
    _raises(lambda: P.conv_nd(**ok, out=m(2, 5, 7, 7, 4)), "x must be a GPU tensor")


def test_conv_nd_activation():
    ok = dict(x=m(*X2), filters=m(*F2), bias=None, g=G2)
    _raises(lambda: P.conv_nd(**ok, act=(AL, (0, 1), m(5, 2), m(5))), "x must be a GPU")
    _raises(lambda: P.conv_nd(**ok, act=(AL, (0, 1), m(3, 2), m(5))), "act weight has shape")
    _raises(lambda: P.conv_nd(**ok, act=(AL, (0, 1), m(5, 3), m(5))), "act weight has shape")
    _raises(lambda: P.conv_nd(**ok, act=(AL, (0, 1), m(5, 2), m(3))), "act bias has shape")
    _raises(lambda: P.conv_nd(**ok, act=(AL, (0, 1), None, m(5))), "needs a weight")
    _raises(lambda: P.conv_nd(**ok, act=(AS, (0, 4), None, None)), "blades")
    _raises(lambda: P.conv_nd(**ok, act=(AS, (1, 1), None, None)), "blades")
    _raises(lambda: P.conv_nd(**ok, act=(AM, (), None, None)), "blades")
    _raises(lambda: P.conv_nd(**ok, act=(7, (0,), None, None)), "aggregation mode")
    _raises(lambda: P.conv_nd(**ok, act=(AM, (0, 1, 2, 3), None, None)), "x must be a GPU")


def test_linear_shapes():
    ok = dict(x=m(6, 3, 8), weight=m(3, 4, 8), bias=m(4, 8), g=(1, 1, 1))
    _raises(lambda: P.linear(**ok), "x must be a GPU tensor")
    _raises(lambda: P.linear(**{**ok, "x": m(6, 3, 4)}), "x has shape")
    _raises(lambda: P.linear(**{**ok, "weight": m(2, 4, 8)}), "weight has shape")
    _raises(lambda: P.linear(**{**ok, "bias": m(3, 8)}), "bias has shape")
    _raises(lambda: P.linear(**ok, out=m(6, 3, 8)), "out has shape")
    _raises(lambda: P.linear(**ok, act=(AL, (0,), m(3, 1), m(4))), "act weight has shape")


def test_act_nd_shapes():
    _raises(lambda: P.act_nd(m(2, 3, 5, 4), AL, (0, 1), m(3, 2), m(3)), "x must be a GPU")
    _raises(lambda: P.act_nd(m(2, 3, 5, 3), AS, (0,)), "N_B in")
    _raises(lambda: P.act_nd(m(2, 3), AS, (0,)), "x has shape")
    _raises(lambda: P.act_nd(m(2, 3, 5, 4), AL, (0, 1), m(2, 2), m(3)), "weight has shape")
    _raises(lambda: P.act_nd(m(2, 3, 5, 4), AL, (0, 1), m(3, 2), None), "needs a weight")
    _raises(lambda: P.act_nd(m(2, 3, 5, 4), AS, (0, 9)), "blades")
    _raises(lambda: P.act_nd(m(2, 3, 5, 4), AS, (0,), out=m(2, 3, 4, 4)), "out has shape")


def test_block2_shapes():
    # x [2, 3, 11, 11, 4] -> C_mid 5 (9 x 9) -> C_out 2 (7 x 7)
    x, f1, f2 = m(2, 3, 11, 11, 4), m(3, 5, 3, 3, 4), m(5, 2, 3, 3, 4)
    l1, l2 = (f1, m(5, 4), None), (f2, m(2, 4), (AM, (0, 1, 2, 3), None, None))
    _raises(lambda: P.block2(x, l1, l2, G2), "x must be a GPU tensor")
    _raises(lambda: P.block2(x, l1, (m(4, 2, 3, 3, 4), None, None), G2), "filters2 has shape")
    _raises(lambda: P.block2(x, l1, (m(5, 2, 5, 5, 4), None, None), G2), "filters2 has shape")
    _raises(lambda: P.block2(x, (f1, m(2, 4), None), l2, G2), "bias1 has shape")
    _raises(lambda: P.block2(x, l1, (f2, m(5, 4), None), G2), "bias2 has shape")
    _raises(lambda: P.block2(x, (f1, None, (AL, (0,), m(2, 1), m(2))), l2, G2),
            "act1 weight has shape")
    _raises(lambda: P.block2(x, l1, l2, G2, workspace=m(2, 5, 9, 9, 3)), "workspace holds")
    _raises(lambda: P.block2(x, l1, l2, G2, out=m(2, 2, 9, 9, 4)), "out has shape")
    _raises(lambda: P.block2(m(2, 3, 4, 4, 4), l1, l2, G2), "too small for two layers")
    _raises(lambda: P.block2(x, l1, l2, G2, workspace=m(2, 5, 9, 9, 4), out=m(2, 2, 7, 7, 4)),
            "x must be a GPU tensor")


def test_block_forward_checks_each_layer():
    x = m(2, 3, 9, 9, 4)
    layers = [(m(3, 5, 3, 3, 4), None, None), (m(4, 2, 3, 3, 4), None, None)]
    _raises(lambda: P.block_forward(x, layers[:1], G2), "x must be a GPU tensor")


def test_plans_check_like_the_calls():
    # a plan runs its call's checks once, at construction
    ok = dict(x=m(*X2), filters=m(*F2), bias=m(*B2), g=G2)
    _raises(lambda: P.conv_plan(**ok), "x must be a GPU tensor")
    _raises(lambda: P.conv_plan(**{**ok, "bias": m(4, 4)}), "bias has shape")
    _raises(lambda: P.conv_plan(**ok, out=m(2, 5, 7, 6, 4)), "out has shape")
    _raises(lambda: P.conv_plan(**ok, act=(AL, (0, 1), m(4, 2), m(5))), "act weight has shape")
    x, f1, f2 = m(2, 3, 11, 11, 4), m(3, 5, 3, 3, 4), m(5, 2, 3, 3, 4)
    l1, l2 = (f1, m(5, 4), None), (f2, m(2, 4), None)
    _raises(lambda: P.block2_plan(x, l1, l2, G2), "x must be a GPU tensor")
    _raises(lambda: P.block2_plan(x, l1, (m(4, 2, 3, 3, 4), None, None), G2), "filters2 has shape")
    _raises(lambda: P.block2_plan(x, l1, l2, G2, workspace=m(2, 5, 9, 9, 3)), "workspace holds")
