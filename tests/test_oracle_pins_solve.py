"""Pins of the oracle's solve with the factors (``oracle.solve``,
``oracle.tridiag_skew_solve``): closed forms, the backward error of the
result against X itself, agreement with a general LU solve, exact cases."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import synth


def inv4_closed(X):
    """Closed-form inverse of a 4x4 skew matrix with upper entries
    (a, b, c, d, e, f) = (x01, x02, x03, x12, x13, x23), Pf = af - be + cd:
    X^{-1} = (1/Pf) [[0, -f, e, -d], [f, 0, -c, b], [-e, c, 0, -a], [d, -b, a, 0]]."""
    a, b, c, d, e, f = X[0, 1], X[0, 2], X[0, 3], X[1, 2], X[1, 3], X[2, 3]
    pf = a * f - b * e + c * d
    return np.array([[0, -f, e, -d], [f, 0, -c, b], [-e, c, 0, -a], [d, -b, a, 0]]) / pf


def test_worked_example_inverse_exact():
    X = np.zeros((4, 4))
    X[np.triu_indices(4, 1)] = [1, 2, 3, 4, 5, 6]
    X = X - X.T
    packed, ipiv = oracle.ltlt(X)
    Xi = oracle.solve(packed, ipiv, np.eye(4))
    # Pf = 8: X^{-1} = [[0,-6,5,-4],[6,0,-3,2],[-5,3,0,-1],[4,-2,1,0]] / 8
    ref = np.array([[0, -6, 5, -4], [6, 0, -3, 2], [-5, 3, 0, -1], [4, -2, 1, 0]]) / 8.0
    assert np.abs(Xi - ref).max() <= 1e-15


@pytest.mark.parametrize("seed", range(8))
def test_closed_form_4x4_inverse(seed):
    X = synth.skew_gauss(4, 600 + seed)
    packed, ipiv = oracle.ltlt(X)
    Xi = oracle.solve(packed, ipiv, np.eye(4))
    ref = inv4_closed(X)
    assert np.abs(Xi - ref).max() <= 1e-12 * np.abs(ref).max()


@pytest.mark.parametrize("n", [2, 8, 50])
def test_tridiagonal_recurrences_against_dense_solve(n):
    rng = synth.rng_for(700 + n)
    alpha = rng.standard_normal(n - 1) + np.sign(rng.standard_normal(n - 1)) * 0.5
    T = np.zeros((n, n))
    T[np.arange(1, n), np.arange(n - 1)] = alpha
    T = T - T.T
    R = rng.standard_normal((n, 3))
    W = oracle.tridiag_skew_solve(alpha, R)
    assert np.abs(T @ W - R).max() <= 1e-12 * max(1.0, np.abs(R).max())
    assert np.abs(W - np.linalg.solve(T, R)).max() <= 1e-10 * np.abs(W).max()


def test_tridiagonal_exact_integers():
    # alpha = 1 everywhere: the recurrences only add and subtract integers
    n = 10
    T = np.zeros((n, n))
    T[np.arange(1, n), np.arange(n - 1)] = 1.0
    T = T - T.T
    w = np.arange(1, n + 1, dtype=float) * np.array([1, -1] * (n // 2))
    r = T @ w
    assert np.array_equal(oracle.tridiag_skew_solve(np.ones(n - 1), r), w)


def test_direct_sum_of_2x2_blocks_exact():
    n = 12
    vals = np.arange(1, n // 2 + 1, dtype=float) * 0.5
    X = np.zeros((n, n))
    for i, a in enumerate(vals):
        X[2 * i, 2 * i + 1], X[2 * i + 1, 2 * i] = a, -a
    packed, ipiv = oracle.ltlt(X)
    b = np.arange(1, n + 1, dtype=float)
    x = oracle.solve(packed, ipiv, b)
    ref = np.empty(n)
    ref[0::2] = -b[1::2] / vals                     # [[0, a], [-a, 0]]^{-1} = [[0, -1/a], [1/a, 0]]
    ref[1::2] = b[0::2] / vals
    assert np.array_equal(x, ref)


@pytest.mark.parametrize("n", [50, 200, 600])
def test_backward_error(n):
    X = synth.skew_gauss(n, 800 + n)
    B = synth.rng_for(801 + n).standard_normal((n, 2))
    packed, ipiv = oracle.ltlt(X)
    x = oracle.solve(packed, ipiv, B)
    eps = np.finfo(np.float64).eps
    for c in range(2):
        be = np.abs(X @ x[:, c] - B[:, c]).max() / (np.abs(X).sum(1).max() * np.abs(x[:, c]).max() * n * eps)
        assert be <= 10, be


def test_matches_lu_solve():
    n = 120
    X = synth.skew_gauss(n, 900)
    B = synth.rng_for(901).standard_normal(n)
    packed, ipiv = oracle.ltlt(X)
    x = oracle.solve(packed, ipiv, B)
    ref = np.linalg.solve(X, B)
    cond = np.linalg.cond(X)
    assert np.abs(x - ref).max() <= 100 * cond * np.finfo(float).eps * np.abs(ref).max()


def test_several_right_hand_sides_equal_single_ones():
    n = 40
    X = synth.skew_gauss(n, 902)
    B = synth.rng_for(903).standard_normal((n, 4))
    packed, ipiv = oracle.ltlt(X)
    xs = oracle.solve(packed, ipiv, B)
    for c in range(4):                              # trsm and trsv may round differently
        one = oracle.solve(packed, ipiv, B[:, c])
        assert np.abs(xs[:, c] - one).max() <= 1e-13 * np.abs(one).max()


def test_odd_order_is_singular():
    X = synth.skew_gauss(5, 904)
    packed, ipiv = oracle.ltlt(X)
    with pytest.raises(ValueError):
        oracle.solve(packed, ipiv, np.ones(5))
