"""GPU tests of the pivot rule's tie paths and of non-finite input.

Exact ties (``tie_inputs``): equal magnitudes where the first position is held
by a later lane, wave or workgroup than a tied competitor, equal high 32 bits
with different low bits, and small-integer matrices (many exact ties in the
first steps).  The pivots must match the oracle bit for bit through the tied
steps; the remaining steps follow the usual parity rules (a later split only
as a near-tie).  Non-finite input gives unspecified factors, but every call
must return, and no bounded wait may give up."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import compare_factors, device_colmajor, gpu_factor, host_packed
from tie_inputs import batched_case, factor_cases, high_word_case, pair_case, small_integer

pytestmark = pytest.mark.gpu


def lt():
    import paper_2005_06410_amd as m
    return m


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("case", [0, 1, 2])
def test_exchange_then_tie_factor(case, dtype):
    name, X, setter, winner = factor_cases(dtype)[case]
    print(f"[ties] factor {name} {np.dtype(dtype).name}", flush=True)
    packed, ipiv, logabs, sign, _ = gpu_factor(X.astype(dtype), nb=128)
    assert ipiv[1] == setter and ipiv[2] == winner, (name, ipiv[:4])
    info = compare_factors(X.astype(dtype), packed, ipiv, dtype)
    assert info["first_pivot_mismatch"] >= 3


@pytest.mark.parametrize("case", [0, 1, 2])
def test_exchange_then_tie_complex(case):
    name, X, setter, winner = factor_cases(np.complex128)[case]
    print(f"[ties] complex {name}", flush=True)
    flat, A = device_colmajor(X)
    ip = lt().factor(A, nb=128)
    torch.cuda.synchronize()
    lt().device_status()
    ipiv = ip.cpu().numpy()
    assert ipiv[1] == setter and ipiv[2] == winner, (name, ipiv[:4])
    packed = host_packed(flat, X.shape[0], X.shape[0])
    info = compare_factors(X, packed, ipiv, np.complex128)
    assert info["first_pivot_mismatch"] >= 3


def test_high_word_tie():
    X, winner = high_word_case()
    print("[ties] high-word", flush=True)
    packed, ipiv, logabs, sign, _ = gpu_factor(X, nb=128)
    assert ipiv[1] == winner
    compare_factors(X, packed, ipiv, np.float64)


def test_pair_panel_tie():
    X, setter, winner = pair_case()
    print("[ties] pair panel", flush=True)
    ref_l, ref_s, ref_a, ref_i = oracle.pfaffian_direct(X)
    flat, A = device_colmajor(X)
    ip, logabs, sign = lt().pfaffian_direct(A, nb=128)
    torch.cuda.synchronize()
    lt().device_status()
    ipiv = ip.cpu().numpy()
    assert ipiv[1] == setter and ipiv[3] == winner
    assert np.array_equal(ipiv, ref_i)
    assert int(sign.item()) == ref_s
    assert abs(float(logabs.item()) - ref_l) <= 1e-9 * max(abs(ref_l), 1.0)


def test_batched_tie_and_integers():
    X, setter, winner = batched_case()
    ints = [small_integer(64, 700 + b) for b in range(63)]
    Xs = np.stack([X] + ints)
    print("[ties] batched", flush=True)
    ref_p, ref_i, ref_l, ref_s = oracle.ltlt_batched(Xs)
    buf = np.ascontiguousarray(np.transpose(Xs, (0, 2, 1)))
    d = torch.from_numpy(buf).cuda()
    A = d.as_strided((64, 64, 64), (64 * 64, 1, 64))
    ipiv, logabs, sign = lt().factor_batched(A)
    torch.cuda.synchronize()
    gi = ipiv.cpu().numpy()
    assert gi[0, 1] == setter and gi[0, 2] == winner
    got = np.tril(np.transpose(d.cpu().numpy(), (0, 2, 1)), -1)
    for b in range(64):
        info = compare_factors(Xs[b], got[b], gi[b], np.float64, ref=(ref_p[b], ref_i[b]))
        assert info["first_pivot_mismatch"] >= 3


@pytest.mark.parametrize("n", [300, 1030])
def test_small_integer_factor(n):
    X = small_integer(n, 900 + n)
    print(f"[ties] integers n={n}", flush=True)
    _, _, best, _, rmag = oracle.ltlt_trace(X, nsteps=6)
    ties = int(np.count_nonzero(best[:6] == rmag[:6]))
    assert ties >= 2
    packed, ipiv, logabs, sign, _ = gpu_factor(X, nb=128)
    info = compare_factors(X, packed, ipiv, np.float64)
    assert info["first_pivot_mismatch"] >= 6          # through the exactly tied first steps
    assert oracle.residual(X, packed, ipiv) <= 10


@pytest.mark.parametrize("n", [300, 1030])
def test_small_integer_pfaffian_direct(n):
    X = small_integer(n, 910 + n)
    print(f"[ties] integers direct n={n}", flush=True)
    ref_l, ref_s, _, ref_i = oracle.pfaffian_direct(X)
    flat, A = device_colmajor(X)
    ip, logabs, sign = lt().pfaffian_direct(A, nb=128)
    torch.cuda.synchronize()
    lt().device_status()
    ipiv = ip.cpu().numpy()
    d = np.nonzero(ipiv != ref_i)[0]
    assert len(d) == 0 or d[0] >= 7, d[:3]
    if len(d) == 0:
        assert int(sign.item()) == ref_s
        if ref_s:
            assert abs(float(logabs.item()) - ref_l) <= 1e-9 * max(abs(ref_l), 1.0)


def test_small_integer_complex():
    X = small_integer(300, 920, dtype=np.complex128)
    print("[ties] integers complex", flush=True)
    flat, A = device_colmajor(X)
    ip = lt().factor(A, nb=128)
    torch.cuda.synchronize()
    lt().device_status()
    packed = host_packed(flat, 300, 300)
    info = compare_factors(X, packed, ip.cpu().numpy(), np.complex128)
    assert info["first_pivot_mismatch"] >= 4


# --------------------------------------------------------------------------
# non-finite input: unspecified results, but every call returns and no
# bounded wait gives up (indices never come from values)

def _poisoned(n, seed, dtype=np.float64):
    X = (synth.skew_gauss_complex(n, seed) if np.dtype(dtype).kind == "c" else synth.skew_gauss(n, seed)).astype(dtype)
    X[n // 2, 17] = np.nan
    X[17, n // 2] = np.nan
    X[n - 3, 3] = np.inf
    X[3, n - 3] = -np.inf
    return X


@pytest.mark.parametrize("dtype", [np.float64, np.float32, np.complex128])
def test_nonfinite_factor_terminates(dtype):
    n = 1030
    X = _poisoned(n, 61, dtype)
    print(f"[nonfinite] factor {np.dtype(dtype).name}", flush=True)
    flat, A = device_colmajor(X)
    ip = lt().factor(A, nb=128)
    out = lt().pfaffian(A, ip)
    torch.cuda.synchronize()
    lt().device_status()                                 # no wait gave up
    ipiv = ip.cpu().numpy()
    assert ipiv[0] == 0 and np.all(ipiv >= np.arange(n)) and np.all(ipiv < n)


def test_nonfinite_pfaffian_direct_and_solve_terminate():
    n = 1030
    X = _poisoned(n, 62)
    print("[nonfinite] direct + solve", flush=True)
    flat, A = device_colmajor(X)
    ip, logabs, sign = lt().pfaffian_direct(A, nb=128)
    torch.cuda.synchronize()
    lt().device_status()
    flat2, A2 = device_colmajor(X)
    ip2 = lt().factor(A2, nb=128)
    B = torch.ones((n, 3), dtype=torch.float64, device="cuda").t().contiguous().t()
    lt().solve(A2, ip2, B)
    torch.cuda.synchronize()
    lt().device_status()


def test_nonfinite_batched_terminates():
    Xs = synth.skew_batch(64, 32, 63)
    Xs[5, 10, 3] = np.nan
    Xs[5, 3, 10] = np.nan
    Xs[9] = np.nan
    print("[nonfinite] batched", flush=True)
    buf = np.ascontiguousarray(np.transpose(Xs, (0, 2, 1)))
    d = torch.from_numpy(buf).cuda()
    A = d.as_strided((32, 64, 64), (64 * 64, 1, 64))
    ipiv, logabs, sign = lt().factor_batched(A)
    torch.cuda.synchronize()
    gi = ipiv.cpu().numpy()
    assert np.all(gi < 64) and np.all(gi >= np.arange(64))
    # untouched members still match the oracle
    ref_p, ref_i, ref_l, ref_s = oracle.ltlt_batched(Xs[:4])
    assert np.array_equal(gi[:4], ref_i)
