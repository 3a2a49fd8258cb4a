"""Pins of the oracle's complex skew-symmetric reduction and Pfaffian
(``oracle.ltlt`` / ``oracle.pfaffian_packed`` on complex128 / complex64):
exact reductions to the real case, closed forms, brute force, det = Pf^2,
the dense similarity-transform form, the residual and the pivot rule."""
from __future__ import annotations

import cmath
import math

import numpy as np
import pytest

import oracle
import synth
from truths import ltlt_dense, pf_closed4, pf_matchings


def pf_of(X):
    packed, ipiv = oracle.ltlt(X)
    la, ph = oracle.pfaffian_packed(packed, ipiv)
    return la, ph


def pf_value(X):
    la, ph = pf_of(X)
    return 0.0 if ph == 0 else math.exp(la) * ph


@pytest.mark.parametrize("n", [2, 5, 64, 200])
def test_real_input_is_the_real_reduction_bitwise(n):
    X = synth.skew_gauss(n, 1300 + n)
    pr, ir = oracle.ltlt(X)
    pc, ic = oracle.ltlt(X.astype(np.complex128))
    assert np.array_equal(ir, ic)
    assert np.array_equal(pc.real, pr)
    assert not np.any(pc.imag)
    lr, sr = oracle.pfaffian_packed(pr, ir)
    lc, phc = oracle.pfaffian_packed(pc, ic)
    assert lc == lr or (math.isinf(lc) and math.isinf(lr))
    assert phc == complex(sr, 0)


@pytest.mark.parametrize("n", [4, 30, 120])
def test_imaginary_input(n):
    """iX: the same pivots and multipliers, alpha times i, Pf times i^(n/2)."""
    X = synth.skew_gauss(n, 1310 + n)
    pr, ir = oracle.ltlt(X)
    pc, ic = oracle.ltlt(1j * X)
    assert np.array_equal(ir, ic)
    sub = np.arange(1, n), np.arange(n - 1)
    assert np.array_equal(pc[sub].imag, pr[sub]) and not np.any(pc[sub].real)
    low = np.tril(np.ones((n, n), bool), -2)
    assert np.array_equal(pc[low].real, pr[low]) and not np.any(pc[low].imag)
    lr, sr = oracle.pfaffian_packed(pr, ir)
    lc, phc = oracle.pfaffian_packed(pc, ic)
    assert lc == lr
    assert phc == sr * (1j ** (n // 2))


@pytest.mark.parametrize("seed", range(6))
def test_closed_form_4x4(seed):
    X = synth.skew_gauss_complex(4, 1320 + seed)
    ref = pf_closed4(X)
    assert abs(pf_value(X) - ref) <= 1e-13 * abs(ref)


@pytest.mark.parametrize("n", [2, 4, 6, 8, 10])
def test_matching_sum_brute_force(n):
    X = synth.skew_gauss_complex(n, 1330 + n)
    ref = pf_matchings(X)
    assert abs(pf_value(X) - ref) <= 1e-12 * abs(ref)


@pytest.mark.parametrize("n", [20, 60, 150])
def test_det_is_pf_squared(n):
    X = synth.skew_gauss_complex(n, 1340 + n)
    la, ph = pf_of(X)
    dsign, dlog = np.linalg.slogdet(X)
    assert abs(2 * la - dlog) <= 1e-10 * abs(dlog)
    assert abs(ph * ph - dsign) <= 1e-9


@pytest.mark.parametrize("n", [3, 9, 40])
def test_dense_similarity_form(n):
    X = synth.skew_gauss_complex(n, 1350 + n)
    packed, ipiv = oracle.ltlt(X)
    alpha, ipd, Ld, _ = ltlt_dense(X)
    assert np.array_equal(ipiv, ipd)
    got_alpha = packed[np.arange(1, n), np.arange(n - 1)]
    assert np.abs(got_alpha - alpha).max() <= 1e-12 * np.abs(alpha).max()
    L, _, _ = oracle.unpack(packed, ipiv)
    assert np.abs(L - Ld).max() <= 1e-12 * max(1.0, np.abs(Ld).max())


@pytest.mark.parametrize("n,dtype", [(50, np.complex128), (200, np.complex128), (400, np.complex128),
                                     (150, np.complex64)])
def test_residual(n, dtype):
    X = synth.skew_gauss_complex(n, 1360 + n, dtype)
    packed, ipiv = oracle.ltlt(X)
    assert oracle.residual(X, packed, ipiv) <= 10


def test_pivot_rule_is_re_plus_im():
    """Column 0 below the diagonal: 5 (modulus 5, |re| + |im| = 5) against
    3 + 4i (modulus 5, |re| + |im| = 7): the pivot search by |re| + |im|
    takes 3 + 4i; 7 against 3 + 4i ties at 7 and the first index wins."""
    X = np.zeros((4, 4), complex)
    X[1, 0], X[2, 0], X[3, 0] = 5, 3 + 4j, 1
    X[2, 1], X[3, 1], X[3, 2] = 0.5, 0.25j, 2
    X = X - X.T
    packed, ipiv = oracle.ltlt(X)
    assert ipiv[1] == 2 and packed[1, 0] == 3 + 4j
    X2 = X.copy()
    X2[1, 0], X2[0, 1] = 7, -7
    packed2, ipiv2 = oracle.ltlt(X2)
    assert ipiv2[1] == 1 and packed2[1, 0] == 7


@pytest.mark.parametrize("seed", range(3))
def test_permutation_similarity(seed):
    n = 12
    X = synth.skew_gauss_complex(n, 1370 + seed)
    q = synth.rng_for(1380 + seed).permutation(n)
    Q = np.eye(n)[q]
    ref = pf_value(X) * round(np.linalg.det(Q))
    assert abs(pf_value(Q @ X @ Q.T) - ref) <= 1e-12 * abs(ref)


def test_power_of_two_scaling_keeps_pivots_and_multipliers():
    n = 30
    X = synth.skew_gauss_complex(n, 1390)
    pr, ir = oracle.ltlt(X)
    ps, is_ = oracle.ltlt(X * 2.0 ** 7)
    assert np.array_equal(ir, is_)
    low = np.tril(np.ones((n, n), bool), -2)
    assert np.array_equal(ps[low], pr[low])
    sub = np.arange(1, n), np.arange(n - 1)
    assert np.array_equal(ps[sub], pr[sub] * 2.0 ** 7)
    la, ph = oracle.pfaffian_packed(pr, ir)
    ls, phs = oracle.pfaffian_packed(ps, is_)
    assert abs(ls - (la + (n // 2) * 7 * math.log(2.0))) <= 1e-13 * abs(ls)
    assert abs(phs - ph) <= 1e-15


def test_swap_is_dense_permutation():
    n = 9
    X = synth.skew_gauss_complex(n, 1395)
    for r, p in [(0, 8), (2, 5), (3, 4)]:
        Q = np.eye(n)
        Q[[r, p]] = Q[[p, r]]
        assert np.array_equal(oracle.swap_indices(X, r, p), Q @ X @ Q.T)


@pytest.mark.parametrize("n", [1, 3, 7])
def test_odd_order(n):
    la, ph = pf_of(synth.skew_gauss_complex(n, 1396))
    assert la == -math.inf and ph == 0


def test_order_two_is_upper_entry():
    X = np.array([[0, 1.5 - 2j], [-1.5 + 2j, 0]])
    la, ph = pf_of(X)
    assert abs(math.exp(la) * ph - (1.5 - 2j)) <= 1e-15 * 2.5
    assert abs(cmath.phase(ph) - cmath.phase(1.5 - 2j)) <= 1e-15
