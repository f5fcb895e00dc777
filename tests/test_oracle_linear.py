"""Pins for the oracle's Clifford linear layer (paper, Algorithm 2):
output[b, co] = sum_ci weight[ci, co] * input[b, ci] + bias[co].

Independent implementations: the layer computed in faithful matrix
representations of the algebra, and the paper's linear baseline construction
(an expanded real weight (C_out N_B, C_in N_B), built here from the matrix
representation, applied with torch.nn.functional.linear in fp64); plus the
hand-derived d = 1 cases of tests/golden/conv_d1.txt, which are linear
layers with B = 1."""
import numpy as np
import pytest
import torch

import oracle
from algebra_reps import GENERATORS, blade_matrices, from_matrix, to_matrix
from test_oracle_conv import _read_conv_d1


def _case(seed, k, B, C_in, C_out):
    rng = np.random.default_rng(seed)
    nb = 1 << k
    return (rng.standard_normal((B, C_in, nb)), rng.uniform(-0.5, 0.5, (C_in, C_out, nb)),
            rng.standard_normal((C_out, nb)))


@pytest.mark.parametrize("g", sorted(GENERATORS), ids=str)
def test_linear_matches_matrix_representation(g):
    k = len(g)
    x, w, b = _case(21, k, 5, 3, 4)
    mats = blade_matrices(g)
    mx, mw = to_matrix(x, mats), to_matrix(w, mats)
    ref = from_matrix(np.einsum("ioab,nibc->noac", mw, mx), mats).real + b[None]
    np.testing.assert_allclose(oracle.linear(x, w, b, g), ref, atol=1e-12)


@pytest.mark.parametrize("g", [(-1,), (1, 1), (1, -1), (-1, -1), (1, 1, 1)], ids=str)
def test_linear_matches_expanded_weight_torch(g):
    k = len(g)
    nb = 1 << k
    x, w, b = _case(22, k, 7, 4, 3)
    mats = blade_matrices(g)
    Wexp = np.zeros((3, nb, 4, nb))
    for j in range(nb):
        ej = np.zeros(nb)
        ej[j] = 1.0
        col = from_matrix(to_matrix(w, mats) @ to_matrix(ej, mats), mats).real  # [C_in, C_out, N_B]
        Wexp[:, :, :, j] = np.transpose(col, (1, 2, 0))
    y = torch.nn.functional.linear(torch.from_numpy(x.reshape(7, 4 * nb)),
                                   torch.from_numpy(Wexp.reshape(3 * nb, 4 * nb))).numpy()
    ref = y.reshape(7, 3, nb) + b[None]
    np.testing.assert_allclose(oracle.linear(x, w, b, g), ref, atol=1e-12)


def test_linear_golden_cases():
    for g, filt, inp, bias, expect in _read_conv_d1():
        nb = 1 << len(g)
        w = np.array(filt).reshape(len(filt), 1, nb)
        x = np.array(inp).reshape(1, len(inp), nb)
        got = oracle.linear(x, w, np.array(bias).reshape(1, nb), g)
        np.testing.assert_array_equal(got.reshape(nb), np.array(expect), err_msg=str(g))


def test_linear_bilinear_and_zero_weight():
    g = (1, -1, 1)
    x, w, b = _case(23, 3, 4, 3, 2)
    x2, w2, _ = _case(24, 3, 4, 3, 2)
    np.testing.assert_allclose(oracle.linear(2 * x - x2, w, None, g),
                               2 * oracle.linear(x, w, None, g) - oracle.linear(x2, w, None, g),
                               atol=1e-12)
    np.testing.assert_allclose(oracle.linear(x, w + 3 * w2, None, g),
                               oracle.linear(x, w, None, g) + 3 * oracle.linear(x, w2, None, g),
                               atol=1e-12)
    np.testing.assert_array_equal(oracle.linear(x, 0 * w, b, g),
                                  np.broadcast_to(b, (4, 2, 8)))
