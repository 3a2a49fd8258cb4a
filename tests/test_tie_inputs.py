"""The tie layouts of ``tie_inputs`` do what they claim on the oracle: the
designed exchanges happen, and each exact tie goes to the first position, so
the GPU tests that use them test the tie rule and not the construction."""
import numpy as np
import pytest

import oracle
from tie_inputs import batched_case, factor_cases, high_word_case, pair_case, small_integer


@pytest.mark.parametrize("dtype", [np.float64, np.float32, np.complex128])
def test_factor_cases_on_oracle(dtype):
    for name, X, setter, winner in factor_cases(dtype):
        _, ipiv = oracle.ltlt(X.astype(dtype, copy=False), nsteps=3)
        assert ipiv[1] == setter and ipiv[2] == winner, name
        # the tie is exact: the column at step 1 holds equal magnitudes at the
        # winner and at the held-back competitor (old row 1, at `setter`)
        pre, _ = oracle.ltlt(X.astype(dtype, copy=False), nsteps=1)
        c = pre[:, 1]
        mag = (np.abs(c.real) + np.abs(c.imag)) if np.iscomplexobj(c) else np.abs(c)
        assert mag[winner] == mag[setter] == mag[2:].max(), name


def test_high_word_case_on_oracle():
    X, winner = high_word_case()
    _, ipiv = oracle.ltlt(X, nsteps=1)
    assert ipiv[1] == winner
    col = np.abs(X[:, 0])
    hi = col.view(np.uint64) >> np.uint64(32)
    tied = np.nonzero(hi == hi[winner])[0]
    assert len(tied) == 5 and np.count_nonzero(col == col[winner]) == 3   # equal high words, 3 exact maxima


def test_pair_case_on_oracle():
    X, setter, winner = pair_case()
    _, _, _, ipiv = oracle.pfaffian_direct(X)
    assert ipiv[1] == setter and ipiv[3] == winner


def test_batched_case_on_oracle():
    X, setter, winner = batched_case()
    _, ipiv = oracle.ltlt(X, nsteps=2)
    assert ipiv[1] == setter and ipiv[2] == winner


def test_small_integer_inputs_tie():
    X = small_integer(300, 41)
    _, ipiv, best, runner, rmag = oracle.ltlt_trace(X)
    assert np.count_nonzero(best[:4] == rmag[:4]) >= 2          # exact ties in the first steps
