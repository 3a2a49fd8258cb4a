"""Pins for the CPU oracle: each test ties it to a fact it does not compute
itself (a hand-derived example, closed forms, brute-force definitions, exact
invariants, a library determinant, an independent dense formulation)."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth
from truths import block_perm, ltlt_dense, pf_closed4, pf_matchings, pf_permutations

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


def _frac(s):
    return float(Fraction(s))


# --- hand-derived worked example ------------------------------------------------

def test_worked_example_4x4():
    g = _golden("ltlt_worked_4x4.txt")
    n = int(g["n"])
    up = [float(x) for x in g["upper"].split()]
    X = np.zeros((n, n))
    X[np.triu_indices(n, 1)] = up
    X = X - X.T
    packed, ipiv = oracle.ltlt(X)
    assert list(ipiv) == [int(x) for x in g["ipiv"].split()]
    for item in g["packed"].split(";"):
        r, c, v = item.split()
        assert packed[int(r), int(c)] == pytest.approx(_frac(v), rel=1e-15, abs=1e-15)
    alpha = [packed[k + 1, k] for k in range(n - 1)]
    assert alpha == pytest.approx([_frac(a) for a in g["alpha"].split()], rel=1e-15)
    logabs, sign = oracle.pfaffian_packed(packed, ipiv)
    assert sign == int(g["sign"])
    assert logabs == pytest.approx(math.log(float(g["pfaffian"])), rel=1e-14)


# --- closed forms ---------------------------------------------------------------

@pytest.mark.parametrize("seed", range(20))
def test_pf_closed_form_4x4(seed):
    X = synth.skew_gauss(4, 100 + seed)
    logabs, sign = oracle.pfaffian(X)
    ref = pf_closed4(X)
    assert sign == int(np.sign(ref))
    assert logabs == pytest.approx(math.log(abs(ref)), rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("a", [1.5, -2.25, 1e-300, -7e200])
def test_pf_2x2_is_upper_entry(a):
    X = np.array([[0.0, a], [-a, 0.0]])
    packed, ipiv = oracle.ltlt(X)
    assert list(ipiv) == [0, 1]
    assert packed[1, 0] == -a          # alpha_0 = X(1,0) = -a, stored as is
    logabs, sign = oracle.pfaffian_packed(packed, ipiv)
    assert sign == (1 if a > 0 else -1)
    assert logabs == pytest.approx(math.log(abs(a)), rel=1e-14)


@pytest.mark.parametrize("n", [1, 3, 5, 9])
def test_pf_odd_n_is_zero(n):
    X = synth.skew_gauss(n, 7)
    logabs, sign = oracle.pfaffian(X)
    assert sign == 0 and logabs == -math.inf


def test_pf_n0_is_one():
    X = np.zeros((0, 0))
    logabs, sign = oracle.pfaffian(X)
    assert sign == 1 and logabs == 0.0


# --- brute-force definitions ------------------------------------------------------

@pytest.mark.parametrize("n", [2, 4, 6, 8, 10])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_pf_brute_force_matchings(n, seed):
    X = synth.skew_gauss(n, 1000 * n + seed)
    ref = pf_matchings(X)
    logabs, sign = oracle.pfaffian(X)
    assert sign == int(np.sign(ref))
    assert logabs == pytest.approx(math.log(abs(ref)), rel=1e-11, abs=1e-11)


@pytest.mark.parametrize("n", [2, 4, 6, 8])
def test_pf_permutation_definition(n):
    X = synth.skew_gauss(n, 77 + n)
    ref = pf_permutations(X)
    assert ref == pytest.approx(pf_matchings(X), rel=1e-12, abs=1e-12)
    logabs, sign = oracle.pfaffian(X)
    assert sign * math.exp(logabs) == pytest.approx(ref, rel=1e-11)


@pytest.mark.parametrize("n", [16, 64, 200])
def test_det_is_pf_squared(n):
    X = synth.skew_gauss(n, 5000 + n)
    logabs, sign = oracle.pfaffian(X)
    s, logdet = np.linalg.slogdet(X)
    assert s == 1.0
    assert 2 * logabs == pytest.approx(logdet, rel=1e-10)


def test_det_is_pf_squared_graded():
    X = synth.skew_graded(120, 4)
    logabs, sign = oracle.pfaffian(X)
    s, logdet = np.linalg.slogdet(X)
    assert 2 * logabs == pytest.approx(logdet, rel=1e-9)


def test_block_diagonal_4x4_product():
    n = 64
    X = synth.skew_blockdiag4(n, 3)
    packed, ipiv = oracle.ltlt(X)
    logabs, sign = oracle.pfaffian_packed(packed, ipiv)
    ref_log, ref_sign = 0.0, 1
    for b in range(n // 4):
        pf = pf_closed4(X[4 * b:4 * b + 4, 4 * b:4 * b + 4])
        ref_log += math.log(abs(pf))
        ref_sign *= int(np.sign(pf))
    assert sign == ref_sign
    assert logabs == pytest.approx(ref_log, rel=1e-12)
    # columns 4b+3 see only zeros below the diagonal: alpha is exactly 0,
    # no exchange, multipliers exactly 0
    for b in range(n // 4 - 1):
        k = 4 * b + 3
        assert packed[k + 1, k] == 0.0
        assert ipiv[k + 1] == k + 1
        assert np.all(packed[k + 2:, k] == 0.0)


def test_direct_sum_of_2x2_blocks_is_exact():
    n = 12
    X = np.zeros((n, n))
    vals = np.arange(1, n // 2 + 1, dtype=float) * 0.75
    for i, a in enumerate(vals):
        X[2 * i, 2 * i + 1] = a
        X[2 * i + 1, 2 * i] = -a
    packed, ipiv = oracle.ltlt(X)
    L, T, perm = oracle.unpack(packed, ipiv)
    assert np.array_equal(perm, np.arange(n))
    assert np.array_equal(L, np.eye(n))
    assert np.array_equal(T, X)


# --- exact invariants -------------------------------------------------------------

@pytest.mark.parametrize("s", [-3, 5])
def test_power_of_two_scaling_bitwise(s):
    X = synth.skew_gauss(96, 31)
    p0, i0 = oracle.ltlt(X)
    p1, i1 = oracle.ltlt(X * 2.0 ** s)
    assert np.array_equal(i0, i1)
    n = X.shape[0]
    sub = np.array([k + 1 for k in range(n - 1)]), np.arange(n - 1)
    assert np.array_equal(p1[sub], p0[sub] * 2.0 ** s)
    mask = np.tril(np.ones((n, n), bool), -2)
    assert np.array_equal(p1[mask], p0[mask])


def test_negation_bitwise():
    X = synth.skew_graded(80, 9)
    p0, i0 = oracle.ltlt(X)
    p1, i1 = oracle.ltlt(-X)
    n = X.shape[0]
    assert np.array_equal(i0, i1)
    sub = np.arange(1, n), np.arange(n - 1)
    assert np.array_equal(p1[sub], -p0[sub])
    mask = np.tril(np.ones((n, n), bool), -2)
    assert np.array_equal(p1[mask], p0[mask])


def test_tridiagonal_input_is_its_own_factor():
    n = 33
    rng = synth.rng_for(12)
    X = np.zeros((n, n))
    d = rng.standard_normal(n - 1)
    d[5] = 0.0
    X[np.arange(1, n), np.arange(n - 1)] = d
    X = X - X.T
    packed, ipiv = oracle.ltlt(X)
    L, T, perm = oracle.unpack(packed, ipiv)
    assert np.array_equal(perm, np.arange(n))
    assert np.array_equal(L, np.eye(n))
    assert np.array_equal(T, X)


@pytest.mark.parametrize("gen", ["gauss", "graded"])
def test_structure_and_pivot_bounds(gen):
    n = 150
    X = synth.skew_gauss(n, 3) if gen == "gauss" else synth.skew_graded(n, 3)
    packed, ipiv = oracle.ltlt(X)
    assert ipiv[0] == 0 and ipiv[n - 1] == n - 1
    assert np.all(ipiv >= np.arange(n))
    L, T, perm = oracle.unpack(packed, ipiv)
    assert np.all(np.abs(L) <= 1.0)                 # partial pivoting bound
    assert np.array_equal(L[:, 0], np.eye(n)[:, 0])
    assert np.all(np.diag(T) == 0) and np.array_equal(T, -T.T)


def test_first_maximum_wins_on_ties():
    # column 0 below the diagonal has |.| = 2 at rows 2 and 4: row 2 must win
    n = 6
    X = np.zeros((n, n))
    X[1, 0], X[2, 0], X[3, 0], X[4, 0], X[5, 0] = 1.0, -2.0, 0.5, 2.0, -1.0
    rng = synth.rng_for(8)
    for i in range(2, n):
        for j in range(1, i):
            X[i, j] = rng.standard_normal()
    X = X - X.T
    packed, ipiv = oracle.ltlt(X)
    assert ipiv[1] == 2


def test_permutation_similarity():
    n = 40
    X = synth.skew_gauss(n, 21)
    rng = synth.rng_for(22)
    q = rng.permutation(n)
    Y = X[np.ix_(q, q)]
    la, sa = oracle.pfaffian(X)
    lb, sb = oracle.pfaffian(Y)
    Q = np.eye(n)[q]
    assert lb == pytest.approx(la, rel=1e-12)
    assert sb == sa * int(round(np.linalg.det(Q)))


@pytest.mark.parametrize("gen,n", [("gauss", 64), ("gauss", 257), ("graded", 200), ("block", 128)])
def test_reconstruction_residual(gen, n):
    X = {"gauss": synth.skew_gauss, "graded": synth.skew_graded, "block": synth.skew_blockdiag4}[gen](n, 11)
    packed, ipiv = oracle.ltlt(X)
    assert oracle.residual(X, packed, ipiv) <= 10.0


def test_reconstruction_residual_fp32():
    X = synth.skew_gauss(160, 13).astype(np.float32)
    packed, ipiv = oracle.ltlt(X)
    assert packed.dtype == np.float32
    assert oracle.residual(X, packed, ipiv) <= 10.0


# --- independent dense formulation ------------------------------------------------

@pytest.mark.parametrize("n,gen", [(5, "gauss"), (8, "gauss"), (12, "graded"), (24, "gauss"), (16, "block")])
def test_matches_dense_similarity_transforms(n, gen):
    X = {"gauss": synth.skew_gauss, "graded": synth.skew_graded, "block": synth.skew_blockdiag4}[gen](n, 40 + n)
    packed, ipiv = oracle.ltlt(X)
    alpha, ipiv_d, L_d, R = ltlt_dense(X)
    assert np.array_equal(ipiv, ipiv_d)
    L, T, perm = oracle.unpack(packed, ipiv)
    scale = np.abs(alpha).max()
    assert np.allclose([packed[k + 1, k] for k in range(n - 1)], alpha, rtol=0, atol=1e-12 * scale)
    assert np.allclose(L, L_d, rtol=0, atol=1e-12)
    # the dense reduction leaves a tridiagonal matrix
    off = R - np.triu(np.tril(R, 1), -1)
    assert np.abs(off).max() <= 1e-12 * scale


def test_swap_is_a_symmetric_permutation():
    X = synth.skew_gauss(9, 5)
    for r, p in [(1, 7), (2, 3), (0, 8), (4, 5)]:
        Y = oracle.swap_indices(X, r, p)
        q = np.arange(9)
        q[[r, p]] = q[[p, r]]
        assert np.array_equal(Y, X[np.ix_(q, q)])


# --- the blocked form used on the GPU ------------------------------------------------

@pytest.mark.parametrize("n,j,b,gen", [(40, 0, 8, "gauss"), (60, 9, 16, "graded"), (33, 5, 7, "gauss"),
                                       (48, 3, 12, "block")])
def test_block_update_identity(n, j, b, gen):
    """b unblocked steps from step j equal one update
    S(perm, perm) + Lx Tx Lx^T on the trailing indices >= j+b+1, where
    Lx = [L(:, j+1 .. j+b), carry] and Tx is skew tridiagonal with
    Tx[u, u+1] = alpha_{j+u+1} (u < b-1), Tx[b-1, b] = 1."""
    X = {"gauss": synth.skew_gauss, "graded": synth.skew_graded, "block": synth.skew_blockdiag4}[gen](n, 70 + j)
    pj, _ = oracle.ltlt(X, nsteps=j)
    Sj = pj - pj.T                                     # full skew state after j steps
    pb, ipiv = oracle.ltlt(X, nsteps=j + b)
    t0 = j + b + 1
    Lx = np.zeros((n, b + 1))
    for u in range(b):
        Lx[t0:, u] = pb[t0:, j + u]                    # L(:, j+u+1) = packed column j+u
    Lx[t0:, b] = pb[t0:, j + b]                        # carry: current column j+b
    Tx = np.zeros((b + 1, b + 1))
    for u in range(b):
        a = pb[j + u + 2, j + u + 1] if u < b - 1 else 1.0
        Tx[u, u + 1], Tx[u + 1, u] = a, -a
    B = Lx @ Tx.T
    perm = block_perm(ipiv, j, j + b, n)
    new = oracle.skew_update(Sj, Lx, B, perm)
    ref = pb - pb.T
    scale = np.abs(Sj[t0:, t0:]).max()
    assert np.allclose(new[t0:, t0:], ref[t0:, t0:], rtol=0, atol=1e-12 * scale)
    # the same update written as the two skew rank-b products of the panel steps
    V = np.zeros((n, b))
    for u in range(b - 1):
        V[t0:, u] = Tx[u, u + 1] * Lx[t0:, u + 1]
    V[t0:, b - 1] = Lx[t0:, b]
    two = Sj[np.ix_(perm, perm)] + Lx[:, :b] @ V.T - V @ Lx[:, :b].T
    assert np.allclose(two[t0:, t0:], ref[t0:, t0:], rtol=0, atol=1e-12 * scale)


# --- batched entry -------------------------------------------------------------------

def test_batched_matches_single():
    Xs = synth.skew_batch(10, 6, 606)
    packed, ipiv, logabs, sign = oracle.ltlt_batched(Xs)
    for b in range(6):
        p1, i1 = oracle.ltlt(Xs[b])
        assert np.array_equal(packed[b], p1) and np.array_equal(ipiv[b], i1)
        l1, s1 = oracle.pfaffian_packed(p1, i1)
        assert logabs[b] == l1 and sign[b] == s1
        ref = pf_matchings(Xs[b])
        assert sign[b] == int(np.sign(ref))
        assert logabs[b] == pytest.approx(math.log(abs(ref)), rel=1e-11)


# --- threads and the decision trace ---------------------------------------------

@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_thread_count_does_not_change_bits(dtype):
    # OpenMP splits the rank-2 update's columns: every entry is still formed by
    # the same operations in the same order, so any thread count gives the same
    # bits (checked against one thread, with more threads than columns at the end)
    X = synth.skew_graded(300, 41).astype(dtype)
    old = oracle.get_threads()
    try:
        oracle.set_threads(1)
        p1, i1 = oracle.ltlt(X)
        oracle.set_threads(5)
        p5, i5 = oracle.ltlt(X)
        oracle.set_threads(64)
        p64, i64 = oracle.ltlt(X)
    finally:
        oracle.set_threads(old)
    assert np.array_equal(i1, i5) and np.array_equal(i1, i64)
    assert np.array_equal(p1.view(np.uint8), p5.view(np.uint8))
    assert np.array_equal(p1.view(np.uint8), p64.view(np.uint8))


def test_trace_worked_example():
    # column 0 of the worked example is (-1, -2, -3) below row 0: pivot row 3
    # (|-3|), runner-up row 2 (|-2|); after the exchange and update, column 1
    # below row 1 is (6, 5): pivot row 2, runner-up row 3
    g = _golden("ltlt_worked_4x4.txt")
    X = np.zeros((4, 4))
    X[np.triu_indices(4, 1)] = [float(x) for x in g["upper"].split()]
    X = X - X.T
    packed, ipiv, best, runner, rmag = oracle.ltlt_trace(X)
    assert list(best) == [3.0, 6.0] and list(runner) == [2, 3] and list(rmag) == [2.0, 5.0]
    p0, i0 = oracle.ltlt(X)
    assert np.array_equal(packed, p0) and np.array_equal(ipiv, i0)


@pytest.mark.parametrize("gen", ["gauss", "ints"])
def test_trace_against_columns(gen):
    # brute force: run the oracle k steps, read column k of the partly reduced
    # matrix, and rank its magnitudes with a stable sort (first index first)
    n = 40
    if gen == "gauss":
        X = synth.skew_gauss(n, 77)
    else:
        U = synth.rng_for(78).integers(-2, 3, size=(n, n)).astype(np.float64)
        X = synth.skew_from_upper(U)
    packed, ipiv, best, runner, rmag = oracle.ltlt_trace(X)
    for k in range(n - 2):
        pre, _ = oracle.ltlt(X, nsteps=k)
        col = np.abs(pre[k + 1:, k])
        order = np.argsort(-col, kind="stable")
        assert ipiv[k + 1] == k + 1 + order[0]
        assert best[k] == col[order[0]]
        assert runner[k] == k + 1 + order[1] and rmag[k] == col[order[1]]


def test_trace_smallest_orders():
    # n = 3: one step with candidate rows 1 and 2; n = 2: no step at all
    X = synth.skew_gauss(3, 5)
    _, ipiv, best, runner, rmag = oracle.ltlt_trace(X)
    a1, a2 = abs(X[1, 0]), abs(X[2, 0])
    win, lose = (1, 2) if a1 >= a2 else (2, 1)
    assert ipiv[1] == win and runner[0] == lose
    assert best[0] == max(a1, a2) and rmag[0] == min(a1, a2)
    _, _, best2, runner2, _ = oracle.ltlt_trace(synth.skew_gauss(2, 5))
    assert len(best2) == 0 and len(runner2) == 0
