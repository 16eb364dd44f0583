"""Pins of the oracle's Gram-Schmidt to the textbook thin QR factorisation."""

import numpy as np
import pytest

from oracle.gs import gram_schmidt


def _rand(k, r, seed):
    return np.random.default_rng(seed).standard_normal((k, r))


@pytest.mark.parametrize("k,r,seed", [(12, 3, 0), (50, 4, 1), (200, 32, 2), (7, 7, 3), (576, 4, 4)])
def test_orthonormal_and_triangular(k, r, seed):
    A = _rand(k, r, seed)
    Q = gram_schmidt(A)
    assert np.abs(Q.T @ Q - np.eye(r)).max() < 1e-10
    R = Q.T @ A
    assert np.abs(np.tril(R, -1)).max() < 1e-10          # upper triangular
    assert (np.diag(R) > 0).all()                          # positive diagonal
    assert np.abs(Q @ R - A).max() < 1e-10 * np.abs(A).max()


@pytest.mark.parametrize("k,r,seed", [(30, 5, 5), (300, 32, 6)])
def test_equals_householder_up_to_sign(k, r, seed):
    A = _rand(k, r, seed)
    Qh, Rh = np.linalg.qr(A)
    ref = Qh * np.sign(np.diag(Rh))
    assert np.abs(gram_schmidt(A) - ref).max() < 1e-10


def test_scale_and_triangular_invariance():
    A = _rand(40, 4, 7)
    Q = gram_schmidt(A)
    assert np.abs(gram_schmidt(3.5 * A) - Q).max() < 1e-12
    U = np.triu(np.random.default_rng(8).standard_normal((4, 4)), 1) + np.diag([1.0, 2.0, 0.5, 3.0])
    assert np.abs(gram_schmidt(A @ U) - Q).max() < 1e-10


def test_column_order_matters():
    A = _rand(40, 3, 9)
    Q = gram_schmidt(A)
    # the first column is the normalised first input column
    assert np.allclose(Q[:, 0], A[:, 0] / np.linalg.norm(A[:, 0]), atol=1e-14)
    assert not np.allclose(gram_schmidt(A[:, ::-1])[:, 0], Q[:, 0])


def test_zero_and_dependent_columns():
    A = _rand(20, 4, 10)
    A[:, 1] = 0.0
    A[:, 3] = 2.0 * A[:, 0] - A[:, 2]
    Q = gram_schmidt(A)
    assert np.all(Q[:, 1] == 0) and np.all(Q[:, 3] == 0)
    ref = gram_schmidt(A[:, [0, 2]])
    assert np.abs(Q[:, [0, 2]] - ref).max() < 1e-12
    assert np.all(gram_schmidt(np.zeros((9, 3))) == 0)


def test_nearly_dependent_column_threshold():
    A = _rand(30, 2, 11)
    e = np.random.default_rng(12).standard_normal(30)
    e -= A[:, 0] * (A[:, 0] @ e) / (A[:, 0] @ A[:, 0])
    e /= np.linalg.norm(e)
    base = A[:, 0] / np.linalg.norm(A[:, 0])
    below = np.stack([A[:, 0], base + 0.5e-4 * e], axis=1)
    above = np.stack([A[:, 0], base + 2e-4 * e], axis=1)
    assert np.all(gram_schmidt(below)[:, 1] == 0)
    assert np.abs(gram_schmidt(above)[:, 1] - e).max() < 1e-8
