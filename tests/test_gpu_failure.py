"""Failure path of the bounded device-side waits, forced from the host.

With ``test_force_timeout`` on, every call starts as if one of its waits had
given up: the waits end at their first poll, every kernel still runs to its
end with all accesses in bounds (a panel's unfinished row order is clamped by
its consumers), the results are poisoned (NaN factor columns, log|Pf| NaN and
sign 0) and the sticky flag makes ``device_status`` raise once.  No kernel is
made to wait for long or to fault."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import synth
from gpu_util import compare_factors, device_colmajor, gpu_factor, host_packed

pytestmark = pytest.mark.gpu


def lt():
    import paper_2005_06410_amd as m
    return m


class forced:
    def __enter__(self):
        lt().device_status()                      # start with the sticky flag clear
        lt().test_force_timeout(True)

    def __exit__(self, *exc):
        lt().test_force_timeout(False)
        return False


def expect_timeout():
    with pytest.raises(lt().LtltError) as e:
        lt().device_status()
    assert e.value.code == -3000
    lt().device_status()                          # read once: cleared


@pytest.mark.parametrize("dtype,nb", [(np.float64, 128), (np.float32, 64), (np.float64, 256)])
def test_forced_timeout_factor(dtype, nb):
    n = 1030
    X = synth.skew_gauss(n, 71).astype(dtype)
    print(f"[failure] factor {np.dtype(dtype).name} nb={nb}", flush=True)
    with forced():
        flat, A = device_colmajor(X)
        ip = lt().factor(A, nb=nb)
        logabs, sign = lt().pfaffian(A, ip)
        torch.cuda.synchronize()
    assert math.isnan(float(logabs.item())) and int(sign.item()) == 0
    packed = host_packed(flat, n, n)
    assert np.isnan(np.diag(packed, -1)).all()   # every block's commit poisoned
    ipiv = ip.cpu().numpy()
    assert np.all(ipiv >= np.arange(n)) and np.all(ipiv < n)
    up = np.triu_indices(n, 0)
    assert np.array_equal(flat.cpu().numpy().reshape(n, n).T[up], X[up])   # upper triangle untouched
    expect_timeout()
    # the next call is unaffected
    packed2, ipiv2, _, _, _ = gpu_factor(X, nb=nb)
    compare_factors(X, packed2, ipiv2, dtype)


def test_forced_timeout_is_sticky_across_calls():
    n = 600
    X = synth.skew_gauss(n, 72)
    print("[failure] sticky", flush=True)
    with forced():
        flat, A = device_colmajor(X)
        lt().factor(A, nb=128)
    flat2, A2 = device_colmajor(X)
    ip2 = lt().factor(A2, nb=128)                 # a good call after the failed one
    torch.cuda.synchronize()
    expect_timeout()                              # the failure is still reported
    compare_factors(X, host_packed(flat2, n, n), ip2.cpu().numpy(), np.float64)


def test_forced_timeout_pfaffian_direct_solve_complex():
    n = 1030
    X = synth.skew_gauss(n, 73)
    print("[failure] direct, solve, complex", flush=True)
    with forced():
        flat, A = device_colmajor(X)
        ip, logabs, sign = lt().pfaffian_direct(A, nb=128)
        torch.cuda.synchronize()
    assert math.isnan(float(logabs.item())) and int(sign.item()) == 0
    expect_timeout()

    flat, A = device_colmajor(X)
    ip = lt().factor(A, nb=128)
    B = torch.ones((n, 2), dtype=torch.float64, device="cuda").t().contiguous().t()
    with forced():
        lt().solve(A, ip, B)
        torch.cuda.synchronize()
    expect_timeout()

    Xc = synth.skew_gauss_complex(n, 74)
    with forced():
        flat, A = device_colmajor(Xc)
        ip = lt().factor(A, nb=128)
        logabs, phase = lt().pfaffian(A, ip)
        torch.cuda.synchronize()
    assert math.isnan(float(logabs.item())) and complex(phase.item()) == 0
    expect_timeout()
