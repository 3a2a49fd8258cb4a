"""Seeded synthetic skew-symmetric inputs.

This module only draws random numbers and lays them out; it contains none of
the factorization's arithmetic.  Both the CPU oracle (through the tests) and
the GPU path take their inputs from here, so both see bit-identical matrices.

Conventions
-----------
* A matrix ``X`` is returned as a C-ordered ``numpy`` array with ``X[i, j]``
  meaning row ``i``, column ``j``; ``X.T == -X`` exactly and ``diag(X) == 0``.
* The strict upper triangle holds the independent draws; the strict lower
  triangle is their exact negation.
* ``to_colmajor`` turns such a matrix into the column-major buffer (leading
  dimension ``lda``) that the library reads, following the Fortran storage
  convention the paper adopts for all of its matrices (section 2, "Data
  storage").
* Random streams: ``numpy.random.Philox`` keyed by a ``SeedSequence`` built
  from the seed (and, for batches, the matrix index), so each matrix of a batch
  has its own independent stream.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "rng_for",
    "skew_gauss",
    "skew_graded",
    "skew_blockdiag4",
    "skew_batch",
    "skew_from_upper",
    "to_colmajor",
    "from_colmajor",
]


def rng_for(seed: int, index: int | None = None) -> np.random.Generator:
    """Counter-based generator for ``seed`` (and optional batch ``index``)."""
    key = [int(seed)] if index is None else [int(seed), int(index)]
    return np.random.Generator(np.random.Philox(np.random.SeedSequence(key)))


def skew_from_upper(U: np.ndarray) -> np.ndarray:
    """Skew matrix whose strict upper triangle is that of ``U``."""
    T = np.triu(U, 1)
    X = T - T.T
    return X


def skew_gauss(n: int, seed: int, dtype=np.float64) -> np.ndarray:
    """Strict-upper entries iid N(0,1); lower = -upper; zero diagonal."""
    rng = rng_for(seed)
    G = rng.standard_normal((n, n))
    X = skew_from_upper(G)
    return X.astype(dtype, copy=False)


def skew_gauss_complex(n: int, seed: int, dtype=np.complex128) -> np.ndarray:
    """Complex skew-symmetric (X^T = -X, no conjugation): strict-upper real and
    imaginary parts iid N(0,1); lower = -upper; zero diagonal."""
    rng = rng_for(seed)
    G = rng.standard_normal((2, n, n))
    X = skew_from_upper(G[0] + 1j * G[1])
    return X.astype(dtype, copy=False)


def skew_graded(n: int, seed: int, dtype=np.float64, decades: float = 3.0) -> np.ndarray:
    """Strict-upper entries N(0,1) * 10**U(-decades, decades), elementwise.

    The graded magnitudes make the pivot order matter: a wrong pivot choice
    produces multipliers far above 1.
    """
    rng = rng_for(seed)
    G = rng.standard_normal((n, n))
    E = rng.uniform(-decades, decades, size=(n, n))
    X = skew_from_upper(G * np.power(10.0, E))
    return X.astype(dtype, copy=False)


def skew_blockdiag4(n: int, seed: int, dtype=np.float64) -> np.ndarray:
    """Direct sum of n/4 Gaussian skew 4x4 blocks (n must be a multiple of 4)."""
    if n % 4:
        raise ValueError("n must be a multiple of 4")
    rng = rng_for(seed)
    X = np.zeros((n, n))
    for b in range(n // 4):
        g = rng.standard_normal(6)
        blk = np.zeros((4, 4))
        blk[0, 1], blk[0, 2], blk[0, 3], blk[1, 2], blk[1, 3], blk[2, 3] = g
        blk = blk - blk.T
        X[4 * b:4 * b + 4, 4 * b:4 * b + 4] = blk
    return X.astype(dtype, copy=False)


def skew_batch(n: int, batch: int, seed: int, dtype=np.float64) -> np.ndarray:
    """``batch`` independent Gaussian skew n x n matrices, shape (batch, n, n).

    Matrix ``i`` draws from its own stream keyed by (seed, i).
    """
    out = np.empty((batch, n, n), dtype=np.float64)
    iu = np.triu_indices(n, 1)
    for i in range(batch):
        g = rng_for(seed, i).standard_normal(len(iu[0]))
        M = np.zeros((n, n))
        M[iu] = g
        out[i] = M - M.T
    return out.astype(dtype, copy=False)


def to_colmajor(X: np.ndarray, lda: int | None = None, fill=0.0) -> np.ndarray:
    """Column-major buffer of ``X``: returns an array ``buf`` of shape (n, lda)
    (C order) with ``buf[c, i] = X[i, c]`` for i < n; padding rows get ``fill``.

    ``buf.ravel()`` is exactly the memory the library reads with leading
    dimension ``lda``.
    """
    n = X.shape[0]
    lda = n if lda is None else int(lda)
    if lda < max(1, n):
        raise ValueError("lda must be >= max(1, n)")
    buf = np.full((n, lda), fill, dtype=X.dtype)
    buf[:, :n] = X.T
    return buf


def from_colmajor(buf: np.ndarray, n: int) -> np.ndarray:
    """Inverse of ``to_colmajor``: the n x n matrix stored in ``buf``."""
    return np.ascontiguousarray(buf[:, :n].T)
