"""The comparison rule of the GPU tests, checked on the CPU with the oracle's
own factors standing in for the GPU's: untouched factors pass, and planted
mistakes (one multiplier or one subdiagonal entry off, a pivot that is not a
near-tie) fail.  For fp32 the fp64-anchored acceptance is exercised on both
sides of its bound, 4 max(d, n eps32), d the fp32 oracle's distance from the
fp64 factors."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import TOL, compare_factors


def _factor(n, seed, dtype):
    X = synth.skew_gauss(n, seed).astype(dtype)
    return X, oracle.ltlt(X)


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_oracle_factors_pass(dtype):
    X, (P, ipiv) = _factor(96, 3, dtype)
    info = compare_factors(X, P.copy(), ipiv, dtype)
    assert info["L_err"] == 0.0 and info["alpha_err"] == 0.0


@pytest.mark.parametrize("where", ["L", "alpha", "last_alpha"])
def test_planted_fp64_mistake_fails(where):
    n = 64
    X, (P, ipiv) = _factor(n, 5, np.float64)
    bad = P.copy()
    i, j = {"L": (n - 1, 3), "alpha": (20, 19), "last_alpha": (n - 1, n - 2)}[where]
    bad[i, j] += 1e-8 * np.abs(P).max()
    with pytest.raises(AssertionError):
        compare_factors(X, bad, ipiv, np.float64)


def test_non_tie_pivot_fails():
    n = 64
    X, (P, ipiv) = _factor(n, 9, np.float64)
    k = 10
    pre, _ = oracle.ltlt(X, nsteps=k - 1)
    col = np.abs(pre[:, k - 1])
    col[:k] = np.inf                               # only rows below the step are candidates
    other = int(np.argmin(col))                    # the smallest candidate: far from a tie
    assert other != ipiv[k]
    bad_ipiv = ipiv.copy()
    bad_ipiv[k] = other
    with pytest.raises(AssertionError, match="near-tie"):
        compare_factors(X, P.copy(), bad_ipiv, np.float64)


@pytest.mark.parametrize("part", ["L", "alpha"])
def test_fp32_anchored_acceptance(part):
    """At n = 300 the bound 4 n eps32 (1.43e-4) exceeds the first bar (1e-4),
    so a result off the fp32 oracle by more than 1e-4 but within the bound of
    the fp64 factors passes, and one beyond the bound fails."""
    n = 300
    X, (P32, ipiv) = _factor(n, 7, np.float32)
    P64, i64 = oracle.ltlt(X.astype(np.float64))
    assert np.array_equal(i64, ipiv)
    low = np.tril(np.ones((n, n), bool), -2)
    sub = np.arange(1, n), np.arange(n - 1)
    ne = n * float(np.finfo(np.float32).eps)
    if part == "L":
        i, j = n - 1, 0
        d = np.abs(P32[low].astype(np.float64) - P64[low]).max()
        scale = np.abs(P64[low]).max()
    else:
        i, j = 150, 149
        d = np.abs(P32[sub].astype(np.float64) - P64[sub]).max() / np.abs(P64[sub]).max()
        scale = np.abs(P64[sub]).max()
    bound = 4.0 * max(d, ne)
    first = max(TOL[np.float32], 2.0 * d)
    assert bound > 1.2 * first                     # the two bars are apart at this size
    side = 1.0 if P64[i, j] >= P32[i, j] else -1.0   # move away from the fp32 oracle
    for frac, ok in ((0.5 * (first + bound) / bound, True), (1.5, False)):
        S = P64.copy()
        S[i, j] += side * frac * bound * scale
        S = S.astype(np.float32)
        if ok:
            info = compare_factors(X, S, ipiv, np.float32)
            assert f"{part}_err_exact" in info     # passed through the anchored branch
        else:
            with pytest.raises(AssertionError, match="from fp64"):
                compare_factors(X, S, ipiv, np.float32)


def _split_case():
    """Graded fp32 input on which the fp32 and fp64 oracles choose different
    pivots at step 377 (a near-tie that rounding decides)."""
    X = synth.skew_graded(800, 1).astype(np.float32)
    P32, i32 = oracle.ltlt(X)
    P64, i64 = oracle.ltlt(X.astype(np.float64))
    return X, P32, i32, P64, i64


def test_fp32_oracle_split_compares_prefix():
    X, P32, i32, P64, i64 = _split_case()
    info = compare_factors(X, P32.copy(), i32, np.float32)
    assert info["oracle_split"] == 378 and info["first_pivot_mismatch"] == 800
    # the fp64 oracle's factors, rounded, with its own pivots: a near-tie
    # split at the same step, accepted, prefix within the bars
    info = compare_factors(X, P64.astype(np.float32), i64, np.float32)
    assert info["first_pivot_mismatch"] == 378


def test_fp32_oracle_split_planted_mistake_fails():
    X, P32, i32, P64, i64 = _split_case()
    bad = P32.copy()
    bad[600, 100] += 1e-2 * np.abs(P32[:, :377]).max()    # a multiplier of step 100, before the split
    with pytest.raises(AssertionError):
        compare_factors(X, bad, i32, np.float32)
    bad = P32.copy()
    bad[201, 200] *= 1.01                                    # alpha_200
    with pytest.raises(AssertionError):
        compare_factors(X, bad, i32, np.float32)
