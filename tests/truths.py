"""Facts that pin the oracle, computed without it.

Nothing here imports the oracle or the GPU library.

* ``pf_closed4``      -- the closed-form 4x4 Pfaffian x01 x23 - x02 x13 + x03 x12.
* ``pf_matchings``    -- the Pfaffian as the signed sum over perfect matchings
                         (expansion along the first row), exact for n <= 10.
* ``pf_permutations`` -- the Pfaffian from its permutation-sum definition
                         1/(2^m m!) sum_sigma sgn(sigma) prod_i x_{sigma(2i) sigma(2i+1)},
                         n = 2m <= 8.
* ``ltlt_dense``      -- the pivoted reduction written as explicit full-matrix
                         similarity transforms X <- M Q X Q^T M^T with dense
                         permutation and Gauss matrices (no packed storage, no
                         lower-triangle bookkeeping).
* ``block_perm``      -- composition of the exchanges of a range of steps.
"""
from __future__ import annotations

import itertools
import math

import numpy as np


def pf_closed4(X) -> float:
    return X[0, 1] * X[2, 3] - X[0, 2] * X[1, 3] + X[0, 3] * X[1, 2]


def pf_matchings(X) -> float:
    """Signed sum over perfect matchings (recursive first-row expansion);
    complex input gives a complex sum."""
    X = np.asarray(X, dtype=np.complex128 if np.iscomplexobj(X) else np.float64)

    def rec(idx):
        if not idx:
            return 1.0
        if len(idx) % 2:
            return 0.0
        i0, rest = idx[0], idx[1:]
        total = 0.0
        for pos, j in enumerate(rest):
            sign = -1.0 if pos % 2 else 1.0
            sub = rest[:pos] + rest[pos + 1:]
            total += sign * X[i0, j] * rec(sub)
        return total

    return rec(tuple(range(X.shape[0])))


def _perm_sign(p) -> int:
    p = list(p)
    s = 1
    seen = [False] * len(p)
    for i in range(len(p)):
        if seen[i]:
            continue
        j, length = i, 0
        while not seen[j]:
            seen[j] = True
            j = p[j]
            length += 1
        if length % 2 == 0:
            s = -s
    return s


def pf_permutations(X) -> float:
    X = np.asarray(X, dtype=np.float64)
    n = X.shape[0]
    if n % 2:
        return 0.0
    m = n // 2
    total = 0.0
    for p in itertools.permutations(range(n)):
        prod = 1.0
        for i in range(m):
            prod *= X[p[2 * i], p[2 * i + 1]]
        total += _perm_sign(p) * prod
    return total / (2 ** m * math.factorial(m))


def ltlt_dense(X):
    """Explicit full-matrix form of the pivoted reduction.

    Returns (alpha, ipiv, L, R) where R is the final reduced matrix (which is
    tridiagonal up to rounding), ipiv the exchanges (first maximum wins), and
    L the unit lower factor with rows in final order, built as
    L = P (M_last ... M_0 P_0^T ... )^{-1}-style accumulation: here simply
    by carrying each multiplier column through the later exchanges.
    """
    cplx = np.iscomplexobj(X)
    dt = np.complex128 if cplx else np.float64
    A = np.array(X, dtype=dt)
    n = A.shape[0]
    ipiv = np.arange(n)
    cols = []                      # multiplier vectors, full length n
    alpha = []
    for k in range(max(n - 2, 0)):
        # complex: the magnitude of the BLAS complex i_amax, |re| + |im|
        col = np.abs(A[k + 1:, k].real) + np.abs(A[k + 1:, k].imag) if cplx else np.abs(A[k + 1:, k])
        p = k + 1 + int(np.argmax(col))            # argmax returns the first maximum
        if col.max() == 0:
            p = k + 1
        ipiv[k + 1] = p
        Q = np.eye(n)
        Q[[k + 1, p]] = Q[[p, k + 1]]
        A = Q @ A @ Q.T
        for c in cols:                              # carry earlier multipliers along
            c[[k + 1, p]] = c[[p, k + 1]]
        a = A[k + 1, k]
        alpha.append(a)
        l = np.zeros(n, dtype=dt)
        if a != 0:
            l[k + 2:] = A[k + 2:, k] / a
        cols.append(l)
        M = np.eye(n, dtype=dt)
        M[k + 2:, k + 1] = -l[k + 2:]
        A = M @ A @ M.T
    if n >= 2:
        alpha.append(A[n - 1, n - 2])
    L = np.eye(n, dtype=dt)
    for k, l in enumerate(cols):
        L[k + 2:, k + 1] = l[k + 2:]
    return np.array(alpha), ipiv, L, A


def block_perm(ipiv, start: int, stop: int, n: int) -> np.ndarray:
    """perm with perm[i] = index held at block start by current index i after
    the exchanges of steps start .. stop-1 (exchange of step k: (k+1, ipiv[k+1]))."""
    perm = np.arange(n)
    for k in range(start, stop):
        a, b = k + 1, int(ipiv[k + 1])
        perm[a], perm[b] = perm[b], perm[a]
    return perm
