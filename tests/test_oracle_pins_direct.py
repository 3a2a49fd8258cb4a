"""Pins of the oracle's Pfaffian by the even column steps only
(``oracle.pfaffian_direct``): each test ties it to a fact outside the oracle
-- a hand-derived example, closed forms, brute-force definitions, det = Pf^2,
exact invariants -- so that a dropped term, a wrong sign or index, or a
skipped update fails one of them."""
from __future__ import annotations

import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth
from truths import pf_closed4, pf_matchings

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            k, v = line.split("=", 1)
            vals[k.strip()] = v.strip()
    return vals


def test_worked_example_4x4():
    g = _golden("pfaffian_direct_worked_4x4.txt")
    n = int(g["n"])
    X = np.zeros((n, n))
    X[np.triu_indices(n, 1)] = [float(x) for x in g["upper"].split()]
    X = X - X.T
    logabs, sign, alpha, ipiv = oracle.pfaffian_direct(X)
    assert list(ipiv) == [int(x) for x in g["ipiv"].split()]
    assert list(alpha) == pytest.approx([float(Fraction(a)) for a in g["alpha_even"].split()], rel=1e-15)
    assert sign == int(g["sign"])
    assert logabs == pytest.approx(math.log(float(g["pfaffian"])), rel=1e-14)


@pytest.mark.parametrize("seed", range(12))
def test_closed_form_4x4(seed):
    X = synth.skew_gauss(4, 300 + seed)
    ref = pf_closed4(X)
    logabs, sign, _, _ = oracle.pfaffian_direct(X)
    assert sign == int(np.sign(ref))
    assert logabs == pytest.approx(math.log(abs(ref)), rel=1e-13, abs=1e-13)


@pytest.mark.parametrize("a", [2.5, -0.125])
def test_2x2_is_upper_entry(a):
    X = np.array([[0.0, a], [-a, 0.0]])
    logabs, sign, alpha, ipiv = oracle.pfaffian_direct(X)
    assert list(alpha) == [-a] and list(ipiv) == [0, 1]
    assert sign == int(np.sign(a)) and logabs == math.log(abs(a))


@pytest.mark.parametrize("n", [1, 3, 7])
def test_odd_n_is_zero(n):
    logabs, sign, alpha, ipiv = oracle.pfaffian_direct(synth.skew_gauss(n, n))
    assert sign == 0 and logabs == -math.inf and len(alpha) == 0
    assert list(ipiv) == list(range(n))


@pytest.mark.parametrize("n", [2, 4, 6, 8, 10])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_brute_force_matchings(n, seed):
    X = synth.skew_gauss(n, 7000 * n + seed)
    ref = pf_matchings(X)
    logabs, sign, _, _ = oracle.pfaffian_direct(X)
    assert sign == int(np.sign(ref))
    assert logabs == pytest.approx(math.log(abs(ref)), rel=1e-11, abs=1e-11)


@pytest.mark.parametrize("n", [16, 64, 200])
def test_det_is_pf_squared(n):
    X = synth.skew_gauss(n, 9000 + n)
    logabs, sign, _, _ = oracle.pfaffian_direct(X)
    s, logdet = np.linalg.slogdet(X)
    assert s == 1.0
    assert 2 * logabs == pytest.approx(logdet, rel=1e-10)


def test_det_is_pf_squared_graded():
    X = synth.skew_graded(120, 14)
    logabs, _, _, _ = oracle.pfaffian_direct(X)
    _, logdet = np.linalg.slogdet(X)
    assert 2 * logabs == pytest.approx(logdet, rel=1e-9)


def test_block_diagonal_4x4_product():
    n = 64
    X = synth.skew_blockdiag4(n, 8)
    logabs, sign, alpha, _ = oracle.pfaffian_direct(X)
    ref_log, ref_sign = 0.0, 1
    for b in range(n // 4):
        pf = pf_closed4(X[4 * b:4 * b + 4, 4 * b:4 * b + 4])
        ref_log += math.log(abs(pf))
        ref_sign *= int(np.sign(pf))
    assert sign == ref_sign
    assert logabs == pytest.approx(ref_log, rel=1e-12)


def test_permutation_similarity():
    # Pf(Q X Q^T) = det(Q) Pf(X) for a permutation Q
    n = 40
    X = synth.skew_gauss(n, 41)
    q = synth.rng_for(42).permutation(n)
    Y = X[np.ix_(q, q)]
    l0, s0, _, _ = oracle.pfaffian_direct(X)
    l1, s1, _, _ = oracle.pfaffian_direct(Y)
    det_q = round(np.linalg.det(np.eye(n)[q]))
    assert s1 == s0 * det_q
    assert l1 == pytest.approx(l0, rel=1e-11)


@pytest.mark.parametrize("s", [-4, 7])
def test_power_of_two_scaling_bitwise(s):
    X = synth.skew_gauss(90, 51)
    l0, s0, a0, i0 = oracle.pfaffian_direct(X)
    l1, s1, a1, i1 = oracle.pfaffian_direct(X * 2.0 ** s)
    assert np.array_equal(i0, i1)
    assert np.array_equal(a1, a0 * 2.0 ** s)
    assert s1 == s0


def test_negation_bitwise():
    X = synth.skew_graded(70, 52)
    l0, s0, a0, i0 = oracle.pfaffian_direct(X)
    l1, s1, a1, i1 = oracle.pfaffian_direct(-X)
    assert np.array_equal(i0, i1)
    assert np.array_equal(a1, -a0)
    assert s1 == s0 * (-1) ** (70 // 2)         # Pf(-X) = (-1)^(n/2) Pf(X)


def test_first_step_is_the_full_first_step():
    # step 0 is the same column step in both methods
    X = synth.skew_gauss(50, 53)
    packed, ipiv_full = oracle.ltlt(X)
    _, _, alpha, ipiv = oracle.pfaffian_direct(X)
    assert ipiv[1] == ipiv_full[1]
    assert alpha[0] == packed[1, 0]


def test_first_maximum_wins_on_ties():
    # column 0 has equal magnitudes at rows 2 and 3 (rows 1 smaller): row 2
    n = 6
    X = synth.skew_gauss(n, 54)
    X[1, 0], X[2, 0], X[3, 0], X[4, 0], X[5, 0] = 0.1, -0.5, 0.5, 0.2, 0.3
    X[0, 1:] = -X[1:, 0]
    _, _, _, ipiv = oracle.pfaffian_direct(X)
    assert ipiv[1] == 2


def test_skew_tridiagonal_needs_no_exchange():
    # tridiagonal skew input: every even step finds its pivot at k+1 and the
    # product of the even subdiagonal entries is the Pfaffian, exactly
    n = 20
    d = synth.rng_for(55).standard_normal(n - 1) + 3.0
    X = np.zeros((n, n))
    X[np.arange(1, n), np.arange(n - 1)] = d
    X = X - X.T
    logabs, sign, alpha, ipiv = oracle.pfaffian_direct(X)
    assert list(ipiv) == list(range(n))
    assert np.array_equal(alpha, d[0::2])
