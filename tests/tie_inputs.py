"""Skew-symmetric inputs with exact pivot ties placed on purpose.

The pivot rule takes the first index of the largest magnitude.  On the GPU a
candidate row lives in a lane chosen by the row's index at the start of the
block, while "first" refers to its current position; after an exchange the two
orders differ.  These inputs put exactly equal magnitudes where the first
position is held by a later lane, wave or workgroup than a tied competitor, so
that a rule "lowest lane / wave / workgroup wins" and the correct rule give
different pivots.

Construction (all values exact): column 0 is zero except X(s, 0) = 5, so step 0
exchanges indices 1 and s and every multiplier of step 0 is exactly 0 -- the
trailing matrix is untouched and step 1 sees column s of X unchanged, its
candidates at the current positions: position s now holds the old row 1.  Column s
carries equal magnitudes at the chosen rows (old row 1 among them, now at
position s) and small Gaussian entries elsewhere; the rest of the matrix is
small Gaussian so that later steps are generic.

Nothing here computes any part of the factorization; the expected winners
follow from the construction and a CPU test confirms them on the oracle.
"""
from __future__ import annotations

import numpy as np

import synth


def _base(n: int, seed: int, scale: float = 0.01, dtype=np.float64) -> np.ndarray:
    if np.dtype(dtype).kind == "c":
        X = synth.skew_gauss_complex(n, seed) * scale
    else:
        X = synth.skew_gauss(n, seed) * scale
    X[:, 0] = 0
    X[0, :] = 0
    return X


def _put(X: np.ndarray, i: int, j: int, v) -> None:
    """X(i, j) = v and X(j, i) = -v."""
    X[i, j] = v
    X[j, i] = -v


def exchange_then_tie(n: int, setter: int, tie_rows, tie_vals, seed: int, dtype=np.float64):
    """Step 0 exchanges 1 and ``setter``; step 1's column is column ``setter``
    of X, whose entries at ``tie_rows`` (old row 1 may be one of them: it sits
    at position ``setter`` after the exchange) are ``tie_vals`` (equal
    magnitudes).  Returns X; the step-1 pivot is the smallest current position
    among the tied rows."""
    X = _base(n, seed, dtype=dtype)
    _put(X, setter, 0, 5.0)
    for r, v in zip(tie_rows, tie_vals):
        _put(X, r, setter, v)
    return X


def step1_position(row: int, setter: int) -> int:
    """Current position at step 1 of the row that started as ``row``."""
    return setter if row == 1 else (1 if row == setter else row)


def factor_cases(dtype=np.float64):
    """(name, X, expected ipiv[1], expected ipiv[2]) for a 1030 x 1030 matrix
    factored with 128-step blocks: two lanes per row, 32 rows per wave, 256 rows
    per workgroup (workgroup w holds block-start indices 1 + 256 w ..)."""
    n = 1030
    cx = dtype if np.dtype(dtype).kind == "c" else None
    if cx is None:
        v = [3.0, -3.0, 3.0]
    else:   # |re| + |im| = 3 for each
        v = [1 + 2j, -3.0, 2 - 1j]
    cases = []
    # the first position (300, workgroup 1) against old row 1 (workgroup 0) at
    # position 700 and row 900 (workgroup 3)
    cases.append(("cross_workgroup", exchange_then_tie(n, 700, [1, 300, 900], v, 31, dtype), 700, 300))
    # same workgroup: position 100 (wave 3) against old row 1 (wave 0) at 250
    cases.append(("cross_wave", exchange_then_tie(n, 250, [1, 100, 240], v, 32, dtype), 250, 100))
    # same wave: position 10 (lane 9) against old row 1 (lane 0) at position 20
    cases.append(("same_wave", exchange_then_tie(n, 20, [1, 10, 25], v, 33, dtype), 20, 10))
    return cases


def high_word_case(n: int = 1030, seed: int = 34):
    """Column 0 holds magnitudes 10 + d 2^-40 (equal high 32 bits, different
    low bits) with mixed signs at rows 5, 9, 40, 300, 1000 (d = 1, 3, 2, 3, 3):
    the pivot is row 9, the first of the largest."""
    X = _base(n, seed)
    rows = [5, 9, 40, 300, 1000]
    d = [1, 3, 2, 3, 3]
    sg = [1, -1, 1, 1, -1]
    for r, dd, s in zip(rows, d, sg):
        if r < n:
            _put(X, r, 0, s * (10.0 + dd * 2.0 ** -40))
    return X, 9


def pair_case(n: int = 1030, seed: int = 35):
    """For the even-step Pfaffian (pair panel, 224 rows per workgroup, 32 per
    working wave): step 0 exchanges 1 and 700 with zero multipliers; step 2's
    column is column 2 of X, with |3| at old row 1 (now at position 700,
    workgroup 0) and at rows 300 (workgroup 1) and 900: the pivot is 300."""
    X = _base(n, seed)
    _put(X, 700, 0, 5.0)
    for r, v in ((1, 3.0), (300, -3.0), (900, 3.0)):
        _put(X, r, 2, v)
    return X, 700, 300


def batched_case(n: int = 64, seed: int = 36):
    """One wave per matrix, lane l holds row l+1: step 0 exchanges 1 and 40;
    step 1 ties old row 1 (lane 0, now at position 40) with row 20 (lane 19)
    and row 50: the pivot is 20."""
    X = exchange_then_tie(n, 40, [1, 20, 50], [3.0, -3.0, 3.0], seed)
    return X, 40, 20


def small_integer(n: int, seed: int, lo: int = -2, hi: int = 2, dtype=np.float64) -> np.ndarray:
    """Strict upper entries uniform integers in [lo, hi]: exact ties in the
    first column steps, then generic rounding."""
    rng = synth.rng_for(seed)
    if np.dtype(dtype).kind == "c":
        U = rng.integers(lo, hi + 1, size=(n, n)) + 1j * rng.integers(lo, hi + 1, size=(n, n))
    else:
        U = rng.integers(lo, hi + 1, size=(n, n)).astype(np.float64)
    return synth.skew_from_upper(U).astype(dtype)
