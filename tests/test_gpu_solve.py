"""GPU parity of the solve with the factors (ltlt_solve) against the oracle's
``solve`` on the same factors, plus the backward error of the GPU solution
against X itself: |X x - b| / (||X|| ||x|| n eps) <= 10."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import device_colmajor

pytestmark = pytest.mark.gpu


def lt():
    import paper_2005_06410_amd as m
    return m


def gpu_factor_solve(X, B, nb=128, dtype=np.float64):
    n = X.shape[0]
    flat, A = device_colmajor(X, dtype=dtype)
    ipiv = lt().factor(A, nb=nb)
    Bd = torch.from_numpy(np.asfortranarray(B.astype(dtype))).cuda()
    if B.ndim == 2:
        Bd = Bd.t().contiguous().t()                 # column-major view
    lt().solve(A, ipiv, Bd)
    torch.cuda.synchronize()
    lt().device_status()
    packed = np.tril(flat.cpu().numpy().reshape(n, n).T, -1)
    return packed, ipiv.cpu().numpy(), Bd.cpu().numpy()


def check(X, B, x, packed, ipiv, tol):
    ref = oracle.solve(packed.astype(np.float64), ipiv, B.astype(np.float64))
    scale = np.abs(ref).max()
    assert np.abs(x.astype(np.float64) - ref).max() <= tol * scale, np.abs(x - ref).max() / scale
    n = X.shape[0]
    eps = np.finfo(x.dtype).eps
    xs = x.reshape(n, -1).astype(np.float64)
    bs = B.reshape(n, -1).astype(np.float64)
    Xd = X.astype(np.float64)
    for c in range(xs.shape[1]):
        be = np.abs(Xd @ xs[:, c] - bs[:, c]).max() / (np.abs(Xd).sum(1).max() * np.abs(xs[:, c]).max() * n * eps)
        assert be <= 10, be


@pytest.mark.parametrize("n,nrhs", [(2, 1), (4, 2), (64, 1), (66, 3), (130, 8), (256, 11), (1000, 1),
                                    (2048, 5)])
def test_parity_fp64(n, nrhs):
    X = synth.skew_gauss(n, 1100 + n)
    B = synth.rng_for(1101 + n).standard_normal((n, nrhs))
    packed, ipiv, x = gpu_factor_solve(X, B)
    check(X, B, x, packed, ipiv, 1e-9)


def test_vector_right_hand_side():
    n = 300
    X = synth.skew_gauss(n, 1200)
    b = synth.rng_for(1201).standard_normal(n)
    packed, ipiv, x = gpu_factor_solve(X, b)
    check(X, b, x, packed, ipiv, 1e-9)


def test_graded_fp64():
    n = 400
    X = synth.skew_graded(n, 1202)
    B = synth.rng_for(1203).standard_normal((n, 2))
    packed, ipiv, x = gpu_factor_solve(X, B, nb=64)
    # graded input: compare with the oracle's solve on the same factors only
    ref = oracle.solve(packed, ipiv, B)
    assert np.abs(x - ref).max() <= 1e-8 * np.abs(ref).max()


def test_closed_form_inverse_4x4():
    X = np.zeros((4, 4))
    X[np.triu_indices(4, 1)] = [1, 2, 3, 4, 5, 6]
    X = X - X.T
    _, _, Xi = gpu_factor_solve(X, np.eye(4))
    ref = np.array([[0, -6, 5, -4], [6, 0, -3, 2], [-5, 3, 0, -1], [4, -2, 1, 0]]) / 8.0
    assert np.abs(Xi - ref).max() <= 1e-15


def test_parity_fp32():
    n = 300
    X = synth.skew_gauss(n, 1204).astype(np.float32)
    B = synth.rng_for(1205).standard_normal((n, 2)).astype(np.float32)
    packed, ipiv, x = gpu_factor_solve(X, B, nb=128, dtype=np.float32)
    check(X, B, x, packed, ipiv, 1e-3)


def test_odd_order_is_refused():
    X = synth.skew_gauss(5, 1206)
    flat, A = device_colmajor(X)
    ipiv = lt().factor(A)
    b = torch.ones(5, dtype=torch.float64, device="cuda")
    with pytest.raises(lt().LtltError):
        lt().solve(A, ipiv, b)


def test_full_size_n16384():
    """The configuration bench.py times: the factors of the n = 16384 Gaussian
    matrix (nb = 128) and one right-hand side: x against the oracle's solve on
    the same factors (normwise 1e-9) and the backward error against X."""
    n = 16384
    X = synth.skew_gauss(n, 5)
    b = synth.rng_for(6).standard_normal((n, 1))
    packed, ipiv, x = gpu_factor_solve(X, b)
    check(X, b, x, packed, ipiv, 1e-9)
