"""MI355X (gfx950) skew-symmetric LTL^T factorization and Pfaffian.

Thin Python binding over the C ABI of ``libltlt.so`` (``include/ltlt.h``):
it only checks layouts and marshals pointers, sizes and the current HIP
stream; every step of the computation runs in the library's gfx950 kernels.
PyTorch supplies device memory and streams.

Matrices are column-major (the Fortran convention): pass a 2-D tensor ``A``
with ``A.stride(0) == 1`` and ``A.stride(1) == lda >= n`` (for example
``torch.empty_strided((n, n), (1, lda), ...)`` or ``X.t().contiguous().t()``),
so that ``A[i, j]`` is element (i, j).  A row-major tensor is rejected: read as
column-major it would be X^T = -X (same L and P, T negated, Pf times
(-1)^(n/2)).

If the library is not built, or no GPU is visible, every call raises; there
is no CPU fallback.

Calls are asynchronous.  ``factor``, ``pfaffian_direct`` and ``solve`` run
device-side waits that are bounded; when one gives up, the results of that
call are poisoned (NaN factor columns, log|Pf| NaN with sign 0) and a sticky
per-device flag is raised.  Pass ``check=True`` to synchronize and raise
``LtltError`` at once, or call ``device_status()`` later: it raises if any
call since the previous ``device_status()`` failed.
"""
from __future__ import annotations

import ctypes
import os
import threading

__all__ = [
    "LIB_PATH",
    "load",
    "factor",
    "pfaffian",
    "factor_batched",
    "skew_update",
    "device_status",
    "test_force_timeout",
    "profile_enable",
    "profile_read",
    "release_workspace",
    "conv_out_size",
    "convgemm",
    "LtltError",
    "F64",
    "F32",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libltlt.so")
F64, F32, C128, C64 = 0, 1, 2, 3
BATCHED_MAX_N = 64
_lock = threading.Lock()
_lib = None

_SYMBOLS = {
    "ltlt_factor": ([ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                     ctypes.c_void_p], ctypes.c_int),
    "ltlt_factor_nb": ([ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                        ctypes.c_int, ctypes.c_void_p], ctypes.c_int),
    "ltlt_pfaffian": ([ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "ltlt_pfaffian_complex": ([ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                               ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "ltlt_factor_batched": ([ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                             ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                             ctypes.c_void_p], ctypes.c_int),
    "ltlt_skew_update": ([ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                          ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                          ctypes.c_void_p], ctypes.c_int),
    "ltlt_device_status": ([ctypes.c_void_p], ctypes.c_int),
    "ltlt_profile_enable": ([ctypes.c_int], ctypes.c_int),
    "ltlt_profile_read": ([ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "ltlt_release_workspace": ([], ctypes.c_int),
    "ltlt_set_cooperative_panels": ([ctypes.c_int], ctypes.c_int),
    "ltlt_mfma_probe": ([ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "ltlt_pfaffian_direct": ([ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                              ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "ltlt_test_force_timeout": ([ctypes.c_int], ctypes.c_int),
    "ltlt_factor_noalloc": ([ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                             ctypes.c_void_p], ctypes.c_int),
    "ltlt_solve": ([ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64,
                    ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p], ctypes.c_int),
    # include/convgemm.h
    "convgemm_out_size": ([ctypes.c_int] * 4, ctypes.c_int),
    "convgemm_f32": ([ctypes.c_int] * 9 + [ctypes.c_void_p] * 3 + [ctypes.c_int] * 4 + [ctypes.c_void_p],
                     ctypes.c_int),
}


class LtltError(RuntimeError):
    """A nonzero return code of the C ABI."""

    def __init__(self, fn: str, code: int):
        self.code = code
        if code <= -3000 and code > -4000:
            what = "a device-side bounded wait gave up"
        elif code == -2000:
            what = "size not supported on this device"
        elif code == -4000:
            what = "X is singular (odd order)"
        elif code == -5000:
            what = "the order needs more than the fixed allocation-free workspace"
        elif code <= -1000:
            what = f"HIP runtime error {-1000 - code}"
        else:
            what = f"argument {-code} is invalid"
        super().__init__(f"{fn} returned {code}: {what}")


def load():
    """Load ``libltlt.so`` (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    f"{LIB_PATH} is missing: build it with `python -m paper_2005_06410_amd.build` "
                    "(the GPU path has no fallback)")
            lib = ctypes.CDLL(LIB_PATH)
            for name, (args, res) in _SYMBOLS.items():
                fn = getattr(lib, name)
                fn.argtypes = args
                fn.restype = res
            _lib = lib
    return _lib


def _check(fn: str, code: int):
    if code != 0:
        raise LtltError(fn, code)


def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float64:
        return F64
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.complex128:
        return C128
    if t.dtype == torch.complex64:
        return C64
    raise TypeError("only float64, float32, complex128 and complex64 are supported")


def _stream_ptr(device) -> int:
    torch = _torch()
    return torch.cuda.current_stream(device).cuda_stream


def _require_gpu(t):
    if not t.is_cuda:
        raise ValueError("tensor must live on a GPU (the library has no CPU path)")


def _same_device(A, *others):
    """Every tensor argument must live on A's GPU: a host or other-device
    pointer handed to a kernel faults the device instead of raising."""
    for t in others:
        if t is not None and (not t.is_cuda or t.device != A.device):
            raise ValueError("all tensor arguments must be on the same GPU as A")


def _check_ipiv(ipiv, n: int):
    torch = _torch()
    if ipiv.dtype != torch.int32 or not ipiv.is_contiguous() or ipiv.numel() < n:
        raise ValueError("ipiv must be a contiguous int32 tensor with at least n entries")


def _colmajor_lda(A) -> int:
    if A.dim() != 2 or A.shape[0] != A.shape[1]:
        raise ValueError("A must be a square 2-D tensor")
    n = A.shape[0]
    if n <= 1:
        return max(1, A.stride(1) if A.dim() == 2 else 1)
    if A.stride(0) != 1 or A.stride(1) < n:
        raise ValueError("A must be column-major: stride(0) == 1 and stride(1) = lda >= n "
                         "(a row-major skew matrix would be read as its negation)")
    return A.stride(1)


def factor(A, ipiv=None, nb: int | None = None, check: bool = False):
    """In-place P X P^T = L T L^T of the column-major skew matrix ``A``
    (float64, float32, or complex128 / complex64 for a complex X with
    X^T = -X).

    Returns the int32 pivot tensor (0-based, LAPACK laswp order).  On return
    A's strict lower triangle holds alpha_k at (k+1, k) and L(r, k+1) at (r, k);
    its strict upper triangle is never touched.  ``check=True`` synchronizes
    and raises if a device-side wait gave up (see the module docstring)."""
    torch = _torch()
    _require_gpu(A)
    lda = _colmajor_lda(A)
    n = A.shape[0]
    if ipiv is None:
        ipiv = torch.empty(max(n, 1), dtype=torch.int32, device=A.device)
    _same_device(A, ipiv)
    _check_ipiv(ipiv, n)
    lib = load()
    s = _stream_ptr(A.device)
    if nb is None:
        code = lib.ltlt_factor(n, A.data_ptr(), lda, _dtype_code(A), ipiv.data_ptr(), s)
    else:
        code = lib.ltlt_factor_nb(n, A.data_ptr(), lda, _dtype_code(A), ipiv.data_ptr(), int(nb), s)
    _check("ltlt_factor", code)
    if check:
        device_status(A.device)
    return ipiv[:n] if ipiv.numel() != n else ipiv


def pfaffian(A, ipiv):
    """(logabs, sign) device tensors of Pf(X) from ``factor``'s output; for a
    complex A, (logabs, phase) with phase = Pf/|Pf| a complex128 tensor."""
    torch = _torch()
    _require_gpu(A)
    lda = _colmajor_lda(A)
    n = A.shape[0]
    _same_device(A, ipiv)
    _check_ipiv(ipiv, n)
    logabs = torch.empty(1, dtype=torch.float64, device=A.device)
    lib = load()
    if A.is_complex():
        phase = torch.empty((1, 2), dtype=torch.float64, device=A.device)
        code = lib.ltlt_pfaffian_complex(n, A.data_ptr(), lda, _dtype_code(A), ipiv.data_ptr(), logabs.data_ptr(),
                                         phase.data_ptr(), _stream_ptr(A.device))
        _check("ltlt_pfaffian_complex", code)
        return logabs, torch.view_as_complex(phase)
    sign = torch.empty(1, dtype=torch.int32, device=A.device)
    code = lib.ltlt_pfaffian(n, A.data_ptr(), lda, _dtype_code(A), ipiv.data_ptr(), logabs.data_ptr(),
                             sign.data_ptr(), _stream_ptr(A.device))
    _check("ltlt_pfaffian", code)
    return logabs, sign


def pfaffian_direct(A, nb: int = 0, ipiv=None, check: bool = False):
    """Pf(X) of the column-major skew matrix ``A`` from the even column steps
    only (see ``ltlt_pfaffian_direct``); ``A`` is used as workspace.

    Returns (ipiv int32 (n,), logabs f64 (1,), sign int32 (1,)) device tensors.
    ``check=True`` synchronizes and raises if a device-side wait gave up."""
    torch = _torch()
    _require_gpu(A)
    lda = _colmajor_lda(A)
    n = A.shape[0]
    if ipiv is None:
        ipiv = torch.empty(max(n, 1), dtype=torch.int32, device=A.device)
    _same_device(A, ipiv)
    _check_ipiv(ipiv, n)
    logabs = torch.empty(1, dtype=torch.float64, device=A.device)
    sign = torch.empty(1, dtype=torch.int32, device=A.device)
    code = load().ltlt_pfaffian_direct(n, A.data_ptr(), lda, _dtype_code(A), ipiv.data_ptr(), int(nb),
                                       logabs.data_ptr(), sign.data_ptr(), _stream_ptr(A.device))
    _check("ltlt_pfaffian_direct", code)
    if check:
        device_status(A.device)
    return ipiv[:n], logabs, sign


def solve(A, ipiv, B, check: bool = False):
    """Overwrite B (column-major n or n x nrhs, same dtype and device as A)
    with X^{-1} B from ``factor``'s output (see ``ltlt_solve``).
    ``check=True`` synchronizes and raises if a device-side wait gave up."""
    _require_gpu(A)
    _require_gpu(B)
    lda = _colmajor_lda(A)
    n = A.shape[0]
    _same_device(A, B, ipiv)
    _check_ipiv(ipiv, n)
    if B.dtype != A.dtype:
        raise ValueError("B must have A's dtype")
    if B.dim() == 1:
        nrhs, ldb = 1, max(B.shape[0], 1)
        if B.stride(0) != 1:
            raise ValueError("B must be contiguous")
    elif B.dim() == 2:
        nrhs = B.shape[1]
        if B.shape[0] > 1 and B.stride(0) != 1:
            raise ValueError("B must be column-major")
        ldb = B.stride(1) if nrhs > 1 else max(B.shape[0], 1)
    else:
        raise ValueError("B must be 1-D or 2-D")
    if B.shape[0] != n:
        raise ValueError("B must have n rows")
    code = load().ltlt_solve(n, A.data_ptr(), lda, _dtype_code(A), ipiv.data_ptr(), nrhs, B.data_ptr(), ldb,
                             _stream_ptr(A.device))
    _check("ltlt_solve", code)
    if check:
        device_status(A.device)
    return B


def factor_batched(A, ipiv=None):
    """Factor and take the Pfaffian of every matrix of a (batch, n, n) tensor
    whose matrices are column-major (``A.stride(1) == 1``, ``A.stride(2) == lda``).

    Returns (ipiv (batch, n) int32, logabs (batch,) f64, sign (batch,) int32)."""
    torch = _torch()
    _require_gpu(A)
    if A.dim() != 3 or A.shape[1] != A.shape[2]:
        raise ValueError("A must be (batch, n, n)")
    batch, n = A.shape[0], A.shape[1]
    if n > 1 and (A.stride(1) != 1 or A.stride(2) < n):
        raise ValueError("each matrix must be column-major: stride(1) == 1, stride(2) = lda >= n")
    lda = A.stride(2) if n > 1 else max(1, n)
    strideA = A.stride(0) if batch > 1 else lda * max(n, 1)
    if ipiv is None:
        ipiv = torch.empty((batch, max(n, 1)), dtype=torch.int32, device=A.device)
    _same_device(A, ipiv)
    if (ipiv.dtype != torch.int32 or ipiv.dim() != 2 or ipiv.shape[0] != batch or ipiv.shape[1] < n
            or (n > 1 and ipiv.stride(1) != 1)):
        raise ValueError("ipiv must be an int32 (batch, >= n) tensor with unit stride along each row")
    logabs = torch.empty(batch, dtype=torch.float64, device=A.device)
    sign = torch.empty(batch, dtype=torch.int32, device=A.device)
    lib = load()
    code = lib.ltlt_factor_batched(n, batch, A.data_ptr(), lda, strideA, _dtype_code(A), ipiv.data_ptr(),
                                   ipiv.stride(0), logabs.data_ptr(), sign.data_ptr(), _stream_ptr(A.device))
    _check("ltlt_factor_batched", code)
    return ipiv[:, :n], logabs, sign


def skew_update(C, Lx, Bt, perm=None, offset: int = 0):
    """The trailing-block update on its own (see ``ltlt_skew_update``).

    ``C`` is a column-major tensor view; the m x m block starting ``offset``
    rows and columns into it is updated; ``perm`` (int32, length m) holds
    source indices relative to that block start."""
    torch = _torch()
    _require_gpu(C)
    if C.dim() != 2 or C.stride(0) != 1:
        raise ValueError("C must be column-major")
    m, K = Lx.shape
    ldc = C.stride(1)
    _same_device(C, Lx, Bt, perm)
    for t in (Lx, Bt):
        if t.dim() != 2 or (t.shape[0] > 1 and t.stride(0) != 1):
            raise ValueError("Lx and Bt must be column-major")
        if t.dtype != C.dtype:
            raise ValueError("Lx and Bt must have C's dtype")
    if tuple(Bt.shape) != (m, K):
        raise ValueError("Bt must have Lx's shape (m, K)")
    if offset < 0 or offset + m > min(C.shape[0], C.shape[1]):
        raise ValueError("the m x m block at `offset` must lie inside C")
    if perm is not None and (perm.dtype != torch.int32 or not perm.is_contiguous() or perm.numel() < m):
        raise ValueError("perm must be a contiguous int32 tensor with at least m entries")
    elem = C.element_size()
    ptr = C.data_ptr() + (offset + offset * ldc) * elem
    pp = 0 if perm is None else perm.data_ptr()

    def ld(t):  # leading dimension; a single column may carry any stride
        return max(t.stride(1), 1) if t.shape[1] > 1 else max(t.shape[0], 1)

    lib = load()
    code = lib.ltlt_skew_update(m, ptr, ldc, pp, K, Lx.data_ptr(), ld(Lx), Bt.data_ptr(), ld(Bt),
                                _dtype_code(C), _stream_ptr(C.device))
    _check("ltlt_skew_update", code)


def conv_out_size(h: int, k: int, stride: int = 1, pad: int = 0) -> int:
    """floor((h - k + 2 pad)/stride) + 1 (``convgemm_out_size``); raises when
    the window does not fit the padded input."""
    r = load().convgemm_out_size(int(h), int(k), int(stride), int(pad))
    if r < 1:
        raise ValueError(f"no output for h={h} k={k} stride={stride} pad={pad}")
    return r


def _leftmost_fastest(t, name):
    """The convolution tensors are stored with the leftmost index fastest."""
    torch = _torch()
    if t.dtype != torch.float32 or t.dim() != 4:
        raise TypeError(f"{name} must be a 4-d float32 tensor")
    if not t.permute(3, 2, 1, 0).is_contiguous():
        raise ValueError(f"{name} must be stored leftmost index fastest (strides (1, d0, d0 d1, d0 d1 d2))")


def convgemm(F, I, stride: int = 1, pad: int = 0, out=None, accumulate: bool = False, path: int = 0,
             tile=(0, 0)):
    """O = conv(F, I) (or O += conv(F, I) with ``accumulate``) by the
    implicit-im2col GEMM of ``convgemm_f32``.

    F: (kn, kh, kw, ci) and I: (hi, wi, ci, b) float32 GPU tensors stored with
    the leftmost index fastest (a numpy Fortran-order array's layout).
    Returns O (kn, ho, wo, b) in the same storage (``out`` if given).
    ``path`` (1 LDS-staged, 2 register-direct) and ``tile`` = (mt, nt) force a
    kernel and workgroup tile (tests and tuning); 0 / (0, 0) choose them."""
    torch = _torch()
    _require_gpu(I)
    _same_device(I, F, out)
    _leftmost_fastest(F, "F")
    _leftmost_fastest(I, "I")
    kn, kh, kw, ci = F.shape
    hi, wi, ci2, b = I.shape
    if ci2 != ci:
        raise ValueError("F and I disagree on the channel count")
    ho, wo = conv_out_size(hi, kh, stride, pad), conv_out_size(wi, kw, stride, pad)
    if out is None:
        flat = torch.empty(max(kn * ho * wo * b, 1), dtype=torch.float32, device=I.device)
        out = flat[:kn * ho * wo * b].as_strided((kn, ho, wo, b), (1, kn, kn * ho, kn * ho * wo))
    else:
        _leftmost_fastest(out, "out")
        if tuple(out.shape) != (kn, ho, wo, b):
            raise ValueError(f"out must have shape {(kn, ho, wo, b)}")
    mt, nt = tile
    code = load().convgemm_f32(kn, kh, kw, ci, hi, wi, b, int(stride), int(pad), F.data_ptr(), I.data_ptr(),
                               out.data_ptr(), int(bool(accumulate)), int(path), int(mt), int(nt),
                               _stream_ptr(I.device))
    _check("convgemm_f32", code)
    return out


def device_status(device=None):
    """Synchronize and raise if a device-side bounded wait of any call on the
    device gave up since the previous ``device_status`` (clears that flag)."""
    torch = _torch()
    lib = load()
    dev = device if device is not None else torch.cuda.current_device()
    with torch.cuda.device(dev):
        _check("ltlt_device_status", lib.ltlt_device_status(_stream_ptr(dev)))


def test_force_timeout(on: bool = True):
    """Failure-path tests only: while on, every factor / pfaffian_direct /
    solve call behaves as if a device-side wait had given up at its start
    (see ``ltlt_test_force_timeout``)."""
    _check("ltlt_test_force_timeout", load().ltlt_test_force_timeout(1 if on else 0))


def profile_enable(on=True):
    """Record per-launch event timings: True (every launch), "update" (the
    trailing-update launches only), or False (stop)."""
    mode = 2 if on == "update" else (1 if on else 0)
    _check("ltlt_profile_enable", load().ltlt_profile_enable(mode))


def profile_read():
    """{kind: (launches, ms, flops)} for kinds panel, update, commit, other."""
    lib = load()
    launches = (ctypes.c_int64 * 4)()
    ms = (ctypes.c_double * 4)()
    flops = (ctypes.c_double * 4)()
    k = lib.ltlt_profile_read(4, launches, ms, flops)
    if k < 0:
        raise LtltError("ltlt_profile_read", k)
    names = ["panel", "update", "commit", "other"]
    return {names[i]: (int(launches[i]), float(ms[i]), float(flops[i])) for i in range(k)}


def release_workspace():
    _check("ltlt_release_workspace", load().ltlt_release_workspace())


def set_cooperative_panels(on: bool = True):
    """Launch the panel kernels with the runtime's cooperative launch (its
    co-residency guarantee, for devices shared with other work) or, the
    default, as ordinary launches (see ``ltlt_set_cooperative_panels``)."""
    _check("ltlt_set_cooperative_panels", load().ltlt_set_cooperative_panels(1 if on else 0))


def mfma_probe(dtype: str = "f64", iters: int = 20000, device=None) -> float:
    """Sustained TFLOP/s of a register-only MFMA loop on the device (see
    ``ltlt_mfma_probe``)."""
    torch = _torch()
    dev = device if device is not None else torch.cuda.current_device()
    out = ctypes.c_double(0.0)
    code = load().ltlt_mfma_probe(0 if dtype == "f64" else 1, int(iters), ctypes.addressof(out), _stream_ptr(dev))
    _check("ltlt_mfma_probe", code)
    return float(out.value)
