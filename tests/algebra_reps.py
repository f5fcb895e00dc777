"""Matrix representations of small Clifford algebras, used to pin the oracle.

Each representation maps the generators e_1..e_k to matrices that satisfy the
defining relations e_i^2 = g_i and e_i e_j = -e_j e_i (paper, Background,
"Clifford Algebra"); a basis blade e_I is the product of its generators in
increasing index order.  The maps below are faithful (the images of the 2^k
blades are linearly independent over the reals), so products and
convolutions computed with matrices and mapped back give an implementation of
the algebra that is independent of the oracle's word-rewriting table.

Blade order: by grade, then lexicographically (the oracle's reading).
"""
from __future__ import annotations

import itertools
from typing import Dict, List, Sequence, Tuple

import numpy as np

I2 = np.eye(2, dtype=complex)
SX = np.array([[0, 1], [1, 0]], dtype=complex)
SY = np.array([[0, -1j], [1j, 0]], dtype=complex)
SZ = np.array([[1, 0], [0, -1]], dtype=complex)
JR = np.array([[0, 1], [-1, 0]], dtype=complex)  # J^2 = -I
NIL = np.array([[0, 1], [0, 0]], dtype=complex)  # N^2 = 0


def blade_words(k: int) -> List[Tuple[int, ...]]:
    words = []
    for grade in range(k + 1):
        words.extend(itertools.combinations(range(1, k + 1), grade))
    return words


def _blkdiag(a, b):
    n, m = a.shape[0], b.shape[0]
    out = np.zeros((n + m, n + m), dtype=complex)
    out[:n, :n] = a
    out[n:, n:] = b
    return out


# generator matrices per signature
GENERATORS: Dict[Tuple[int, ...], List[np.ndarray]] = {
    # complex numbers: e1 -> i
    (-1,): [1j * np.eye(1, dtype=complex)],
    # split-complex numbers: e1 -> sigma_x
    (1,): [SX],
    # dual numbers: e1 -> nilpotent
    (0,): [NIL],
    # Cl(2,0) = M2(R)
    (1, 1): [SZ, SX],
    # Cl(1,1) = M2(R)
    (1, -1): [SZ, JR],
    (-1, 1): [JR, SZ],
    # quaternions: e1 -> i, e2 -> j in the 2x2 complex representation
    (-1, -1): [np.array([[1j, 0], [0, -1j]]), JR],
    # Cl(3,0) = M2(C): Pauli matrices
    (1, 1, 1): [SX, SY, SZ],
    # Cl(0,3) = H + H: e_i -> (q_i, -q_i)
    (-1, -1, -1): [
        _blkdiag(np.array([[1j, 0], [0, -1j]]), -np.array([[1j, 0], [0, -1j]])),
        _blkdiag(JR, -JR),
        _blkdiag(np.array([[0, 1j], [1j, 0]]), -np.array([[0, 1j], [1j, 0]])),
    ],
    # Cl(2,1) = M2(R) + M2(R): e1, e2 -> (sz, -sz), (sx, -sx), e3 -> (J, -J)
    (1, 1, -1): [_blkdiag(SZ, -SZ), _blkdiag(SX, -SX), _blkdiag(JR, -JR)],
    # Cl(1,2) = M2(C): e1 -> sz, e2 -> i sx, e3 -> i sy
    (1, -1, -1): [SZ, 1j * SX, 1j * SY],
}


def blade_matrices(g: Sequence[int]) -> List[np.ndarray]:
    gens = GENERATORS[tuple(g)]
    n = gens[0].shape[0]
    mats = []
    for word in blade_words(len(g)):
        m = np.eye(n, dtype=complex)
        for i in word:
            m = m @ gens[i - 1]
        mats.append(m)
    return mats


def to_matrix(x: np.ndarray, mats: List[np.ndarray]) -> np.ndarray:
    """x [..., N_B] -> [..., n, n] complex."""
    basis = np.stack(mats)  # [N_B, n, n]
    return np.tensordot(np.asarray(x, dtype=complex), basis, axes=([-1], [0]))


def from_matrix(m: np.ndarray, mats: List[np.ndarray]) -> np.ndarray:
    """Inverse of to_matrix (least squares over the real coefficients)."""
    nb = len(mats)
    n = mats[0].shape[0]
    A = np.stack([mm.reshape(-1) for mm in mats], axis=1)  # [n*n, N_B]
    A_real = np.concatenate([A.real, A.imag], axis=0)
    flat = m.reshape(m.shape[:-2] + (n * n,))
    rhs = np.concatenate([flat.real, flat.imag], axis=-1)  # [..., 2 n n]
    pinv = np.linalg.pinv(A_real)  # [N_B, 2 n n]
    return np.tensordot(rhs, pinv, axes=([-1], [1])).reshape(m.shape[:-2] + (nb,))


def is_faithful(mats: List[np.ndarray]) -> bool:
    A = np.stack([m.reshape(-1) for m in mats], axis=1)
    A_real = np.concatenate([A.real, A.imag], axis=0)
    return np.linalg.matrix_rank(A_real) == len(mats)
