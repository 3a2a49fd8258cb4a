"""The seeded generators: determinism, exact skew structure, layouts."""
import numpy as np
import pytest

import synth


@pytest.mark.parametrize("gen", [synth.skew_gauss, synth.skew_graded, synth.skew_blockdiag4])
def test_exact_skew_and_zero_diagonal(gen):
    X = gen(64, 3)
    assert np.array_equal(X.T, -X)
    assert np.all(np.diag(X) == 0)


def test_same_seed_same_bits_different_seed_differs():
    a = synth.skew_gauss(50, 9)
    b = synth.skew_gauss(50, 9)
    c = synth.skew_gauss(50, 10)
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c)


def test_fp32_is_rounded_fp64():
    a = synth.skew_graded(40, 2)
    b = synth.skew_graded(40, 2, dtype=np.float32)
    assert b.dtype == np.float32
    assert np.array_equal(b, a.astype(np.float32))


def test_graded_magnitudes_span_decades():
    X = synth.skew_graded(200, 1)
    a = np.abs(X[np.triu_indices(200, 1)])
    assert a.max() / np.median(a) > 1e2 and np.median(a) / a[a > 0].min() > 1e2


def test_blockdiag_has_no_coupling():
    X = synth.skew_blockdiag4(32, 5)
    mask = np.zeros((32, 32), bool)
    for b in range(8):
        mask[4 * b:4 * b + 4, 4 * b:4 * b + 4] = True
    assert np.all(X[~mask] == 0)


def test_batch_per_matrix_streams():
    A = synth.skew_batch(8, 5, 42)
    B = synth.skew_batch(8, 3, 42)
    assert np.array_equal(A[:3], B)            # matrix i depends only on (seed, i)
    for M in A:
        assert np.array_equal(M.T, -M)
    assert not np.array_equal(A[0], A[1])


def test_colmajor_roundtrip_and_padding():
    X = synth.skew_gauss(7, 4)
    buf = synth.to_colmajor(X, lda=10, fill=np.nan)
    assert buf.shape == (7, 10)
    flat = buf.ravel()
    for i in range(7):
        for j in range(7):
            assert flat[i + j * 10] == X[i, j]
    assert np.all(np.isnan(buf[:, 7:]))
    assert np.array_equal(synth.from_colmajor(buf, 7), X)
    with pytest.raises(ValueError):
        synth.to_colmajor(X, lda=6)
