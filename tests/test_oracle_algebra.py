"""Pins for the oracle's multiplication table (paper, Background, "Clifford
Algebra": e_i^2 = g_i, e_i e_j = -e_j e_i for i != j, e_I the product of its
generators in increasing order).

Two independent pins:
  * matrix representations of ten signatures (complex, split-complex, dual,
    quaternion, M2(R), M2(C), H+H, ...) -- products of the images must match
    the table;
  * for all 39 signatures with k <= 3 (degenerate ones included), the four
    properties that determine the algebra uniquely: the generator relations,
    e_I as an ordered product, unit scalar and associativity.
Plus hand-derived products from tests/golden/blade_products.txt.
"""
import itertools
import os

import numpy as np
import pytest

import oracle
from algebra_reps import GENERATORS, blade_matrices, blade_words, is_faithful

ALL_SIGNATURES = [g for k in (1, 2, 3)
                  for g in itertools.product((-1, 0, 1), repeat=k)]
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_39_signatures():
    assert len(ALL_SIGNATURES) == 39


@pytest.mark.parametrize("g", sorted(GENERATORS), ids=str)
def test_table_matches_matrix_representation(g):
    k = len(g)
    mats = blade_matrices(g)
    assert is_faithful(mats)
    blade, sign = oracle.cayley(k, g)
    for a in range(1 << k):
        for b in range(1 << k):
            lhs = mats[a] @ mats[b]
            rhs = sign[a, b] * mats[blade[a, b]]
            np.testing.assert_allclose(lhs, rhs, atol=1e-12,
                                       err_msg=f"e{a} e{b} in g={g}")


def _product_with_table(blade, sign, x, y):
    nb = blade.shape[0]
    z = np.zeros(nb)
    for a in range(nb):
        for b in range(nb):
            z[blade[a, b]] += sign[a, b] * x[a] * y[b]
    return z


@pytest.mark.parametrize("g", ALL_SIGNATURES, ids=str)
def test_table_is_the_clifford_algebra(g):
    k = len(g)
    nb = 1 << k
    blade, sign = oracle.cayley(k, g)
    words = blade_words(k)
    gen = {words.index((i,)): i for i in range(1, k + 1)}
    # unit scalar
    for a in range(nb):
        assert blade[0, a] == a and sign[0, a] == 1
        assert blade[a, 0] == a and sign[a, 0] == 1
    # generator relations
    for a, i in gen.items():
        for b, j in gen.items():
            if i == j:
                assert blade[a, b] == 0 and sign[a, b] == g[i - 1]
            else:
                assert blade[a, b] == blade[b, a]
                assert sign[a, b] == -sign[b, a]
                assert sign[a, b] in (-1, 1)
    # e_I is the ordered product of its generators
    for idx, word in enumerate(words):
        if len(word) < 2:
            continue
        cur_blade, cur_sign = words.index((word[0],)), 1.0
        for i in word[1:]:
            gb = words.index((i,))
            cur_sign *= sign[cur_blade, gb]
            cur_blade = blade[cur_blade, gb]
        assert cur_blade == idx and cur_sign == 1.0, (word, cur_blade, cur_sign)
    # associativity on random multivectors
    rng = np.random.default_rng(7)
    for _ in range(5):
        x, y, z = rng.standard_normal((3, nb))
        lhs = _product_with_table(blade, sign,
                                  _product_with_table(blade, sign, x, y), z)
        rhs = _product_with_table(blade, sign, x,
                                  _product_with_table(blade, sign, y, z))
        np.testing.assert_allclose(lhs, rhs, atol=1e-12)


def test_blade_square_closed_form():
    # e_I^2 = (-1)^{|I|(|I|-1)/2} prod_{i in I} g_i
    for g in ALL_SIGNATURES:
        k = len(g)
        blade, sign = oracle.cayley(k, g)
        for idx, word in enumerate(blade_words(k)):
            n = len(word)
            expect = (-1) ** (n * (n - 1) // 2) * np.prod([g[i - 1] for i in word])
            assert blade[idx, idx] == 0
            assert sign[idx, idx] == expect, (g, word)


def _read_golden_products():
    rows = []
    with open(os.path.join(GOLDEN, "blade_products.txt")) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            g, a, b, s, c = line.split()
            rows.append((tuple(int(v) for v in g.split(",")), a, b, int(s), c))
    return rows


def _name_to_index(k, name):
    words = blade_words(k)
    if name == "1":
        return 0
    return words.index(tuple(int(ch) for ch in name[1:]))


def test_golden_blade_products():
    rows = _read_golden_products()
    assert len(rows) >= 20
    for g, a, b, s, c in rows:
        k = len(g)
        blade, sign = oracle.cayley(k, g)
        ia, ib = _name_to_index(k, a), _name_to_index(k, b)
        assert sign[ia, ib] == s, (g, a, b)
        if s != 0:
            assert blade[ia, ib] == _name_to_index(k, c), (g, a, b)


def test_hamilton_product():
    # quaternions from i^2 = j^2 = k^2 = ijk = -1, written out component-wise
    def ham(p, q):
        a1, b1, c1, d1 = p
        a2, b2, c2, d2 = q
        return np.array([
            a1 * a2 - b1 * b2 - c1 * c2 - d1 * d2,
            a1 * b2 + b1 * a2 + c1 * d2 - d1 * c2,
            a1 * c2 - b1 * d2 + c1 * a2 + d1 * b2,
            a1 * d2 + b1 * c2 - c1 * b2 + d1 * a2,
        ])
    rng = np.random.default_rng(3)
    for _ in range(10):
        p, q = rng.standard_normal((2, 4))
        np.testing.assert_allclose(oracle.mv_mul(2, (-1, -1), p, q), ham(p, q),
                                   atol=1e-12)


def test_complex_product():
    rng = np.random.default_rng(4)
    for _ in range(10):
        p, q = rng.standard_normal((2, 2))
        z = complex(*p) * complex(*q)
        np.testing.assert_allclose(oracle.mv_mul(1, (-1,), p, q),
                                   [z.real, z.imag], atol=1e-12)
