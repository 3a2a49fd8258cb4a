"""ltlt_factor_noalloc (the entry point for callers that cannot allocate)
against ltlt_factor, through the C ABI: the same kernels on a fixed workspace,
so the factors, pivots and Pfaffian must be bit-identical -- on two calls in a
row, the second one smaller (the fixed array keeps the first call's contents),
in fp64 and fp32, and at the largest order the array serves; one past it is
refused with LTLT_ERR_SCRATCH before anything is enqueued.  The allocation-free
call runs first, so in a fresh process it is also the first call on the device."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import synth
from gpu_util import device_colmajor

pytestmark = pytest.mark.gpu

LTLT_ERR_SCRATCH = -5000
MAX_N = {np.float64: 4928, np.float32: 8128}


def lt():
    import paper_2005_06410_amd as m
    return m


def noalloc(A, ipiv):
    code = {torch.float64: 0, torch.float32: 1, torch.complex128: 2}[A.dtype]
    return noalloc_raw(A.shape[0], A.data_ptr(), A.stride(1), code, ipiv.data_ptr())


def noalloc_raw(n, a_ptr, lda, dtype_code, ipiv_ptr):
    return lt().load().ltlt_factor_noalloc(n, a_ptr, lda, dtype_code, ipiv_ptr,
                                           torch.cuda.current_stream().cuda_stream)


def run_pair(n, dtype, seed):
    X = synth.skew_gauss(n, seed).astype(dtype)
    flat_a, A_a = device_colmajor(X)
    ip_a = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    assert noalloc(A_a, ip_a) == 0
    la_a, sg_a = lt().pfaffian(A_a, ip_a)
    torch.cuda.synchronize()
    lt().device_status()
    flat_b, A_b = device_colmajor(X)
    ip_b = lt().factor(A_b)                        # default width, allocating workspace
    la_b, sg_b = lt().pfaffian(A_b, ip_b)
    torch.cuda.synchronize()
    lt().device_status()
    assert torch.equal(ip_a, ip_b)
    assert torch.equal(flat_a.view(torch.uint8), flat_b.view(torch.uint8))
    assert float(la_a.item()) == float(la_b.item()) and int(sg_a.item()) == int(sg_b.item())


@pytest.mark.parametrize("dtype,sizes", [(np.float64, (1030, 300)), (np.float32, (2000, 257))])
def test_noalloc_matches_factor_twice(dtype, sizes):
    for i, n in enumerate(sizes):
        print(f"[noalloc] {np.dtype(dtype).name} n={n}", flush=True)
        run_pair(n, dtype, 880 + i)


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_noalloc_size_limit(dtype):
    n = MAX_N[dtype]
    print(f"[noalloc] limit {np.dtype(dtype).name} n={n}", flush=True)
    run_pair(n, dtype, 890)
    big = n + 1                                     # refused before anything is enqueued:
    t = torch.empty(1, dtype=torch.float64, device="cuda")  # these buffers are never touched
    ip = torch.empty(1, dtype=torch.int32, device="cuda")
    assert noalloc_raw(big, t.data_ptr(), big, 0 if dtype == np.float64 else 1, ip.data_ptr()) == LTLT_ERR_SCRATCH


def test_noalloc_refuses_complex():
    t = torch.empty(16, dtype=torch.complex128, device="cuda")
    ip = torch.empty(4, dtype=torch.int32, device="cuda")
    assert noalloc_raw(4, t.data_ptr(), 4, 2, ip.data_ptr()) == -4
