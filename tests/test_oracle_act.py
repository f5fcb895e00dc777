"""Pins for the oracle's multivector activation (paper, Algorithm 3): a
scalar gate s computed from K selected blades (Linear: weighted sum plus bias;
Sum; Mean = Sum / K) scales every blade of the multivector by sigmoid(s).

Pins: sigmoid(0) = 1/2 cases, library sigmoid (scipy.special.expit) for the
K = 1 case, the uniform-scaling property, saturation, independence from
blades outside the subset, and folding spatial positions into the batch."""
import numpy as np
import pytest
from scipy.special import expit

import oracle
from workloads import AGG_LINEAR, AGG_MEAN, AGG_SUM, random_act_case


def test_linear_zero_weight_halves():
    x, spec, _, _ = random_act_case(1, 8, 3, 5, 4, AGG_LINEAR, 3)
    w = np.zeros((5, 3))
    b = np.zeros(5)
    out = oracle.act(x, AGG_LINEAR, spec.blades, w, b)
    np.testing.assert_array_equal(out, x.astype(np.float64) * 0.5)


def test_sum_of_opposites_halves():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 3, 5, 4))
    x[..., 2] = -x[..., 0]
    out = oracle.act(x, AGG_SUM, (0, 2))
    np.testing.assert_array_equal(out, x * 0.5)
    out = oracle.act(x, AGG_MEAN, (2, 0))
    np.testing.assert_array_equal(out, x * 0.5)


def test_k1_unit_weight_is_self_gated_blade():
    x, _, _, _ = random_act_case(3, 4, 2, 3, 6, AGG_LINEAR, 1)
    x = x.astype(np.float64)
    for blade in range(4):
        out = oracle.act(x, AGG_LINEAR, (blade,), np.ones((3, 1)), np.zeros(3))
        ref = x * expit(x[..., blade:blade + 1])
        np.testing.assert_allclose(out, ref, rtol=1e-15, atol=0)


@pytest.mark.parametrize("mode", [AGG_LINEAR, AGG_SUM, AGG_MEAN])
def test_uniform_scaling_by_library_sigmoid(mode):
    x, spec, w, b = random_act_case(4, 8, 3, 4, 5, mode, 5)
    x = x.astype(np.float64)
    out = oracle.act(x, mode, spec.blades, w, b)
    ratio = out / x
    # one gate per multivector, the same for all blades, strictly in (0, 1)
    np.testing.assert_allclose(ratio, ratio[..., :1].repeat(8, -1), rtol=1e-14)
    assert np.all((ratio > 0) & (ratio < 1))
    sel = x[..., list(spec.blades)]
    if mode == AGG_LINEAR:
        s = np.einsum("bcpk,ck->bcp", sel, w.astype(np.float64)) + b[None, :, None]
    else:
        s = sel.sum(-1) / (len(spec.blades) if mode == AGG_MEAN else 1)
    np.testing.assert_allclose(ratio[..., 0], expit(s), rtol=1e-13)


def test_sum_and_mean_are_linear_special_cases():
    x, spec, _, _ = random_act_case(5, 8, 2, 3, 4, AGG_SUM, 6)
    K = len(spec.blades)
    lin1 = oracle.act(x, AGG_LINEAR, spec.blades, np.ones((3, K)), np.zeros(3))
    np.testing.assert_array_equal(oracle.act(x, AGG_SUM, spec.blades), lin1)
    linm = oracle.act(x, AGG_LINEAR, spec.blades, np.full((3, K), 1.0 / K),
                      np.zeros(3))
    np.testing.assert_allclose(oracle.act(x, AGG_MEAN, spec.blades), linm,
                               rtol=1e-14)


def test_saturation():
    x = np.ones((1, 2, 1, 4))
    big = oracle.act(x, AGG_LINEAR, (0,), np.array([[800.0], [-800.0]]),
                     np.zeros(2))
    np.testing.assert_array_equal(big[0, 0], x[0, 0])
    np.testing.assert_array_equal(big[0, 1], 0.0 * x[0, 1])


def test_blades_outside_subset_do_not_change_gate():
    x, spec, w, b = random_act_case(6, 8, 2, 3, 4, AGG_LINEAR, 3)
    x = x.astype(np.float64)
    other = [j for j in range(8) if j not in spec.blades][0]
    y = x.copy()
    y[..., other] += 5.0
    ox = oracle.act(x, AGG_LINEAR, spec.blades, w, b)
    oy = oracle.act(y, AGG_LINEAR, spec.blades, w, b)
    keep = [j for j in range(8) if j != other]
    np.testing.assert_array_equal(ox[..., keep], oy[..., keep])


def test_positions_fold_into_batch():
    x, spec, w, b = random_act_case(7, 4, 3, 5, 6, AGG_LINEAR, 4)
    out = oracle.act(x, AGG_LINEAR, spec.blades, w, b)      # [B, C, P, N_B]
    xf = np.ascontiguousarray(np.moveaxis(x, 2, 1)).reshape(18, 5, 4)
    of = oracle.act(xf, AGG_LINEAR, spec.blades, w, b)      # [B P, C, N_B]
    np.testing.assert_array_equal(np.moveaxis(out, 2, 1).reshape(18, 5, 4), of)
