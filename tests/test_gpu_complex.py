"""GPU parity of the complex skew-symmetric factorization (dtype complex128 /
complex64 through ``ltlt_factor``) and its Pfaffian (``ltlt_pfaffian_complex``)
against the complex CPU oracle, on seeded synthetic inputs: pivots compared
bit-exactly as a prefix (a later split only as a near-tie in |re| + |im|),
alpha and L normwise within 1e-10 (complex128), residual <= 10, log|Pf|
within 1e-9 relative and the phase within 1e-9; plus exact structural cases
(real and purely imaginary input) and closed forms."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import compare_factors, device_colmajor, host_packed, residual_probe
from truths import pf_closed4

pytestmark = pytest.mark.gpu


def lt():
    import paper_2005_06410_amd as m
    return m


def gpu_factor_c(X, nb=None, lda=None, fill=0.0):
    n = X.shape[0]
    flat, A = device_colmajor(X, lda=lda, fill=fill)
    ipiv = lt().factor(A, nb=nb)
    logabs, phase = lt().pfaffian(A, ipiv)
    torch.cuda.synchronize()
    lt().device_status()
    packed = host_packed(flat, n, max(lda or n, 1))
    return packed, ipiv.cpu().numpy(), float(logabs.item()), complex(phase.item()), flat


def check_pf(logabs, phase, ref, tol=1e-9):
    rl, rph = ref
    if rph == 0:
        assert logabs == -math.inf and phase == 0
        return
    assert abs(logabs - rl) <= tol * max(abs(rl), 1.0), (logabs, rl)
    assert abs(phase - rph) <= tol, (phase, rph)


def complex_graded(n, seed):
    return synth.skew_graded(n, seed) + 1j * synth.skew_graded(n, seed + 1)


@pytest.mark.parametrize("n,nb", [(3, 1), (4, 1), (5, 2), (8, 3), (17, 4), (33, 8), (64, 16), (100, 32),
                                  (129, 64), (200, 64), (255, 7), (300, 128), (513, 64), (700, 128)])
def test_parity_gauss_c128(n, nb):
    X = synth.skew_gauss_complex(n, 2100 + n)
    packed, ipiv, logabs, phase, _ = gpu_factor_c(X, nb=nb)
    info = compare_factors(X, packed, ipiv, np.complex128)
    assert info["first_pivot_mismatch"] == n
    assert oracle.residual(X, packed, ipiv) <= 10
    check_pf(logabs, phase, oracle.pfaffian(X))


def test_default_block_width():
    X = synth.skew_gauss_complex(260, 2099)
    packed, ipiv, logabs, phase, _ = gpu_factor_c(X)
    compare_factors(X, packed, ipiv, np.complex128)
    check_pf(logabs, phase, oracle.pfaffian(X))


@pytest.mark.parametrize("n,nb", [(64, 8), (400, 64)])
def test_parity_graded_c128(n, nb):
    X = complex_graded(n, 2200 + n)
    packed, ipiv, logabs, phase, _ = gpu_factor_c(X, nb=nb)
    compare_factors(X, packed, ipiv, np.complex128)
    assert oracle.residual(X, packed, ipiv) <= 10
    check_pf(logabs, phase, oracle.pfaffian(X))


@pytest.mark.parametrize("n,nb", [(50, 16), (257, 64), (600, 128)])
def test_parity_c64(n, nb):
    X = synth.skew_gauss_complex(n, 2300 + n, np.complex64)
    packed, ipiv, logabs, phase, _ = gpu_factor_c(X, nb=nb)
    compare_factors(X, packed, ipiv, np.complex64)
    assert oracle.residual(X, packed, ipiv) <= 10
    # complex64 factors: the Pfaffian against the complex128 oracle on the same rounded input
    check_pf(logabs, phase, oracle.pfaffian(X.astype(np.complex128)), tol=1e-4)


def test_real_input_keeps_zero_imaginary_parts():
    """Real data stored as complex: every imaginary part the reduction forms
    is an exact zero, and the factors are the real path's up to rounding."""
    n = 300
    X = synth.skew_gauss(n, 2400)
    packed, ipiv, logabs, phase, _ = gpu_factor_c(X.astype(np.complex128), nb=64)
    assert not np.any(packed.imag)
    compare_factors(X, np.ascontiguousarray(packed.real), ipiv, np.float64)
    rl, rs = oracle.pfaffian(X)
    assert phase == complex(rs, 0)
    assert abs(logabs - rl) <= 1e-9 * abs(rl)


def test_imaginary_input_structure():
    """iX: alphas purely imaginary, multipliers real (exact zeros), the
    factors those of X times i where the oracle says so."""
    n = 260
    X = 1j * synth.skew_gauss(n, 2410)
    packed, ipiv, logabs, phase, _ = gpu_factor_c(X, nb=64)
    sub = np.arange(1, n), np.arange(n - 1)
    low = np.tril(np.ones((n, n), bool), -2)
    assert not np.any(packed[sub].real)
    assert not np.any(packed[low].imag)
    compare_factors(X, packed, ipiv, np.complex128)
    check_pf(logabs, phase, oracle.pfaffian(X))


def test_block_diagonal_closed_forms():
    n = 1024
    rng = synth.rng_for(2420)
    X = np.zeros((n, n), complex)
    for b in range(n // 4):
        g = rng.standard_normal(6) + 1j * rng.standard_normal(6)
        blk = np.zeros((4, 4), complex)
        blk[0, 1], blk[0, 2], blk[0, 3], blk[1, 2], blk[1, 3], blk[2, 3] = g
        X[4 * b:4 * b + 4, 4 * b:4 * b + 4] = blk - blk.T
    packed, ipiv, logabs, phase, _ = gpu_factor_c(X, nb=64)
    ref_log, ref_ph = 0.0, 1.0 + 0j
    for b in range(n // 4):
        pf = pf_closed4(X[4 * b:4 * b + 4, 4 * b:4 * b + 4])
        ref_log += math.log(abs(pf))
        ref_ph *= pf / abs(pf)
    assert abs(logabs - ref_log) <= 1e-9 * abs(ref_log)
    assert abs(phase - ref_ph) <= 1e-9
    for b in range(n // 4 - 1):                     # zero columns: no exchange, alpha and multipliers 0
        k = 4 * b + 3
        assert packed[k + 1, k] == 0 and ipiv[k + 1] == k + 1
        assert np.all(packed[k + 2:, k] == 0)


def test_config_n2048_nb64_det():
    n = 2048
    X = synth.skew_gauss_complex(n, 2430)
    packed, ipiv, logabs, phase, _ = gpu_factor_c(X, nb=64)
    compare_factors(X, packed, ipiv, np.complex128)
    dsign, dlog = np.linalg.slogdet(X)
    assert abs(2 * logabs - dlog) <= 1e-9 * abs(dlog)
    assert abs(phase * phase - dsign) <= 1e-8
    check_pf(logabs, phase, oracle.pfaffian(X))


def test_full_size_sampled():
    """n = 8192 complex128 at the default width: the first column steps
    against the oracle run for those steps only, the residual by random
    probes, and the Pfaffian's modulus against the probes' determinant-free
    reading log|Pf| = sum log|alpha_2j| recomputed on the host."""
    n, steps = 8192, 3
    X = synth.skew_gauss_complex(n, 2440)
    packed, ipiv, logabs, phase, _ = gpu_factor_c(X)
    pre, ipre = oracle.ltlt(X, nsteps=steps)
    assert np.array_equal(ipiv[:steps + 1], ipre[:steps + 1])
    from gpu_util import carry_rows
    ref_cols = carry_rows(pre[:, :steps], ipiv, steps, n)
    got = packed[:, :steps]
    mask = np.tril(np.ones((n, steps), bool), -1)
    err = np.abs(got[mask] - ref_cols[mask]).max() / np.abs(ref_cols[mask]).max()
    assert err <= 1e-10, err
    assert residual_probe(X, packed, ipiv) <= 10
    alpha = packed[np.arange(1, n, 2), np.arange(0, n - 1, 2)]
    assert abs(logabs - float(np.sum(np.log(np.abs(alpha))))) <= 1e-9 * abs(logabs)


@pytest.mark.parametrize("n", [0, 1, 2])
def test_tiny_orders(n):
    X = synth.skew_gauss_complex(n, 2450) if n else np.zeros((0, 0), complex)
    flat, A = device_colmajor(X) if n else (None, torch.zeros((0, 0), dtype=torch.complex128, device="cuda"))
    ipiv = lt().factor(A)
    logabs, phase = lt().pfaffian(A, ipiv)
    torch.cuda.synchronize()
    if n == 0:
        assert float(logabs.item()) == 0.0 and complex(phase.item()) == 1
    elif n == 1:
        assert float(logabs.item()) == -math.inf and complex(phase.item()) == 0
    else:
        assert list(ipiv.cpu().numpy()) == [0, 1]
        assert abs(float(logabs.item()) - math.log(abs(X[0, 1]))) <= 1e-15
        assert abs(complex(phase.item()) - X[0, 1] / abs(X[0, 1])) <= 1e-15


def test_padded_lda_and_untouched_upper_triangle():
    n, lda = 150, 157
    X = synth.skew_gauss_complex(n, 2460)
    flat, A = device_colmajor(X, lda=lda, fill=complex(7.0, -3.0))
    before = flat.cpu().numpy().reshape(n, lda)
    ipiv = lt().factor(A, nb=32)
    torch.cuda.synchronize()
    lt().device_status()
    after = flat.cpu().numpy().reshape(n, lda)
    up = np.triu(np.ones((n, n), bool), 0).T            # buf[c, i] with i <= c: diagonal and upper triangle
    assert np.array_equal(after[:, :n][up], before[:, :n][up])
    assert np.all(after[:, n:] == complex(7.0, -3.0))
    packed = np.ascontiguousarray(np.tril(after[:, :n].T, -1))
    compare_factors(X, packed, ipiv.cpu().numpy(), np.complex128)
