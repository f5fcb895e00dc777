"""Pins for the oracle's Clifford convolution (paper, Algorithm 1).

Independent implementations the oracle must agree with:
  * the convolution computed in a faithful matrix representation of the
    algebra (complex numbers, quaternions, M2(R), M2(C), H+H, ...);
  * the paper's baseline construction: an expanded real kernel
    (C_out N_B, C_in N_B, d_filter^k) fed to torch's real convolution in fp64,
    with the expansion built from the matrix representation;
  * numpy complex correlation for g = (-1);
and closed-form invariants: scalar-only filters, a unit centre tap,
bilinearity, zero filters, translation equivariance, d_image = d_filter = 1
products worked out by hand (tests/golden/conv_d1.txt).
"""
import itertools
import os

import numpy as np
import pytest
import torch

import oracle
from algebra_reps import GENERATORS, blade_matrices, from_matrix, to_matrix
from workloads import random_conv_case

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _shifted(x, q, d_out):
    """x[:, :, q0:q0+d_out, q1:q1+d_out, ...] for spatial axes 2..2+k."""
    sl = (slice(None), slice(None)) + tuple(slice(qi, qi + d_out) for qi in q)
    return x[sl]


def conv_by_matrices(g, x, f, bias):
    k = len(g)
    mats = blade_matrices(g)
    mx = to_matrix(x, mats)          # [B, C_in, d^k, n, n]
    mf = to_matrix(f, mats)          # [C_in, C_out, d_f^k, n, n]
    d_f = f.shape[2]
    d_out = x.shape[2] - d_f + 1
    acc = 0
    for q in itertools.product(range(d_f), repeat=k):
        wq = mf[(slice(None), slice(None)) + q]       # [C_in, C_out, n, n]
        xq = _shifted(mx, q, d_out)                   # [B, C_in, d_out^k, n, n]
        # out[b, co, p] += W[ci, co] @ X[b, ci, p]  (filter on the left)
        acc = acc + np.einsum("ioab,ni...bc->no...ac", wq, xq)
    out = from_matrix(acc, mats)
    if bias is not None:
        out = out + bias.reshape((1, bias.shape[0]) + (1,) * k + (bias.shape[1],))
    return out.real if np.iscomplexobj(out) else out


def expanded_kernel(g, f):
    """(C_out N_B, C_in N_B, d_f^k) real kernel: block (co, ci, q) is the
    left-multiplication matrix of f[ci, co, q], computed in the matrix
    representation."""
    k = len(g)
    nb = 1 << k
    mats = blade_matrices(g)
    C_in, C_out = f.shape[:2]
    taps = f.shape[2:-1]
    K = np.zeros((C_out, nb, C_in, nb) + taps)
    for j in range(nb):
        ej = np.zeros(nb)
        ej[j] = 1.0
        # column j of L_w: coefficients of w * e_j
        prod = to_matrix(f, mats) @ to_matrix(ej, mats)
        col = from_matrix(prod, mats).real                # [C_in, C_out, taps, N_B]
        K[:, :, :, j] = np.moveaxis(col, (0, 1, -1), (2, 0, 1))
    return K.reshape((C_out * nb, C_in * nb) + taps)


def conv_by_torch_expanded(g, x, f, bias):
    k = len(g)
    nb = 1 << k
    B, C_in = x.shape[:2]
    C_out = f.shape[1]
    W = torch.from_numpy(expanded_kernel(g, f))
    # input (B, C_in, d^k, N_B) -> (B, C_in N_B, d^k)
    xt = torch.from_numpy(np.moveaxis(x.astype(np.float64), -1, 2).copy())
    xt = xt.reshape((B, C_in * nb) + x.shape[2:-1])
    conv = {1: torch.nn.functional.conv1d, 2: torch.nn.functional.conv2d,
            3: torch.nn.functional.conv3d}[k]
    y = conv(xt, W).numpy()
    y = y.reshape((B, C_out, nb) + y.shape[2:])
    y = np.moveaxis(y, 2, -1)
    if bias is not None:
        y = y + bias.reshape((1, C_out) + (1,) * k + (nb,))
    return y


MATRIX_CASES = [
    ((-1,), 2, 3, 2, 9, 3),
    ((1,), 2, 2, 3, 8, 2),
    ((0,), 1, 2, 2, 7, 3),
    ((1, 1), 2, 3, 2, 7, 3),
    ((1, -1), 1, 2, 3, 6, 2),
    ((-1, 1), 1, 2, 2, 6, 3),
    ((-1, -1), 2, 2, 3, 7, 3),
    ((1, 1, 1), 1, 2, 2, 5, 3),
    ((-1, -1, -1), 1, 2, 3, 4, 2),
    ((1, 1, -1), 1, 3, 2, 4, 3),
    ((1, -1, -1), 2, 2, 2, 4, 2),
]


@pytest.mark.parametrize("g,B,C_in,C_out,d_img,d_f", MATRIX_CASES, ids=str)
def test_conv_matches_matrix_representation(g, B, C_in, C_out, d_img, d_f):
    assert tuple(g) in GENERATORS
    s, x, f, b = random_conv_case(11, len(g), g, B, C_in, C_out, d_img, d_f)
    ref = conv_by_matrices(g, x.astype(np.float64), f.astype(np.float64),
                           b.astype(np.float64))
    got = oracle.conv_nd(x, f, b, g, nthreads=3)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-11)


@pytest.mark.parametrize("g,d_img,d_f", [((-1,), 11, 4), ((1, 1), 9, 3),
                                         ((1, -1), 8, 2), ((1, 1, 1), 6, 3),
                                         ((-1, -1), 7, 5)], ids=str)
def test_conv_matches_expanded_kernel_torch(g, d_img, d_f):
    s, x, f, b = random_conv_case(12, len(g), g, 2, 3, 2, d_img, d_f)
    ref = conv_by_torch_expanded(g, x, f.astype(np.float64),
                                 b.astype(np.float64))
    got = oracle.conv_nd(x, f, b, g)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-11)


def test_complex_correlation_numpy():
    s, x, f, b = random_conv_case(13, 1, (-1,), 3, 2, 3, 12, 4)
    xc = x[..., 0].astype(np.float64) + 1j * x[..., 1]
    fc = f[..., 0].astype(np.float64) + 1j * f[..., 1]
    d_out = s.d_out
    ref = np.zeros((3, 3, d_out), complex)
    for q in range(4):
        ref += np.einsum("io,bip->bop", fc[:, :, q], xc[:, :, q:q + d_out])
    ref += (b[:, 0] + 1j * b[:, 1])[None, :, None]
    got = oracle.conv_nd(x, f, b, (-1,))
    np.testing.assert_allclose(got[..., 0], ref.real, atol=1e-12)
    np.testing.assert_allclose(got[..., 1], ref.imag, atol=1e-12)


@pytest.mark.parametrize("g", [(1, 1), (0, 1), (1, 1, 1), (-1, 0, 1)], ids=str)
def test_scalar_filter_is_real_conv_per_blade(g):
    k = len(g)
    s, x, f, b = random_conv_case(14, k, g, 2, 3, 2, 7, 3)
    f[..., 1:] = 0.0
    got = oracle.conv_nd(x, f, b, g)
    conv = {2: torch.nn.functional.conv2d, 3: torch.nn.functional.conv3d}[k]
    W = torch.from_numpy(np.moveaxis(f[..., 0], 0, 1).astype(np.float64).copy())
    for i in range(s.nb):
        xi = torch.from_numpy(x[..., i].astype(np.float64).copy())
        ref = conv(xi, W).numpy() + b[None, :, i].reshape((1, -1) + (1,) * k)
        np.testing.assert_allclose(got[..., i], ref, atol=1e-12)


@pytest.mark.parametrize("g,d_f", [((1, 1), 3), ((1, -1, 1), 3), ((-1, -1), 5),
                                   ((0, 1, 1), 1)], ids=str)
def test_unit_centre_tap_crops_input(g, d_f):
    k = len(g)
    s, x, f, b = random_conv_case(15, k, g, 2, 3, 3, 9, d_f)
    f[...] = 0.0
    c = (d_f - 1) // 2
    for ch in range(3):
        f[(ch, ch) + (c,) * k + (0,)] = 1.0
    got = oracle.conv_nd(x, f, None, g)
    crop = (slice(None), slice(None)) + (slice(c, c + s.d_out),) * k
    np.testing.assert_array_equal(got, x[crop].astype(np.float64))


def test_bilinearity():
    g = (1, -1, 1)
    s, x1, f1, _ = random_conv_case(16, 3, g, 2, 2, 2, 5, 2)
    _, x2, f2, _ = random_conv_case(17, 3, g, 2, 2, 2, 5, 2)
    a, c = 0.75, -1.5
    x1, x2, f1, f2 = (v.astype(np.float64) for v in (x1, x2, f1, f2))
    lhs = oracle.conv_nd(a * x1 + c * x2, f1, None, g)
    rhs = a * oracle.conv_nd(x1, f1, None, g) + c * oracle.conv_nd(x2, f1, None, g)
    np.testing.assert_allclose(lhs, rhs, atol=1e-12)
    lhs = oracle.conv_nd(x1, a * f1 + c * f2, None, g)
    rhs = a * oracle.conv_nd(x1, f1, None, g) + c * oracle.conv_nd(x1, f2, None, g)
    np.testing.assert_allclose(lhs, rhs, atol=1e-12)


def test_zero_filter_gives_bias():
    g = (1, 1)
    s, x, f, b = random_conv_case(18, 2, g, 2, 3, 4, 6, 3)
    f[...] = 0.0
    got = oracle.conv_nd(x, f, b, g)
    np.testing.assert_array_equal(
        got, np.broadcast_to(b[None, :, None, None, :], got.shape).astype(np.float64))


def test_translation_equivariance():
    g = (1, 1, -1)
    s, x, f, b = random_conv_case(19, 3, g, 1, 2, 2, 8, 3)
    full = oracle.conv_nd(x, f, b, g)
    head = oracle.conv_nd(x[:, :, 2:, 2:, 2:], f, b, g)
    np.testing.assert_array_equal(head, full[:, :, 2:, 2:, 2:])
    tail = oracle.conv_nd(x[:, :, :-1, :-1, :-1], f, b, g)
    np.testing.assert_array_equal(tail, full[:, :, :-1, :-1, :-1])


def test_points_equal_full_and_threads_invariant():
    g = (1, 1, 1)
    s, x, f, b = random_conv_case(20, 3, g, 2, 3, 2, 6, 3)
    full1 = oracle.conv_nd(x, f, b, g, nthreads=1)
    full5 = oracle.conv_nd(x, f, b, g, nthreads=5)
    np.testing.assert_array_equal(full1, full5)
    rng = np.random.default_rng(0)
    n = 40
    bs = rng.integers(0, 2, n)
    cos = rng.integers(0, 2, n)
    ps = rng.integers(0, s.d_out ** 3, n)
    pts = oracle.conv_points(x, f, b, g, bs, cos, ps)
    flat = full1.reshape(2, 2, -1, 8)
    np.testing.assert_array_equal(pts, flat[bs, cos, ps])


def _read_conv_d1():
    cases = []
    with open(os.path.join(GOLDEN, "conv_d1.txt")) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            fields = line.split("|")
            g = tuple(int(v) for v in fields[0].split(","))
            parse = lambda s: [[float(v) for v in mv.split()] for mv in s.split(";")]
            cases.append((g, parse(fields[1]), parse(fields[2]),
                          [float(v) for v in fields[3].split()],
                          [float(v) for v in fields[4].split()]))
    return cases


def test_golden_d1_convolutions():
    cases = _read_conv_d1()
    assert len(cases) >= 4
    for g, filt, inp, bias, expect in cases:
        k = len(g)
        nb = 1 << k
        C_in = len(filt)
        f = np.array(filt).reshape((C_in, 1) + (1,) * k + (nb,))
        x = np.array(inp).reshape((1, C_in) + (1,) * k + (nb,))
        b = np.array(bias).reshape(1, nb)
        got = oracle.conv_nd(x, f, b, g).reshape(nb)
        np.testing.assert_array_equal(got, np.array(expect), err_msg=str(g))
