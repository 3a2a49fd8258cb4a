"""CPU oracle for the skew-symmetric LTL^T factorization and its Pfaffian.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The GPU library
never links, imports or calls it, and it shares no code with the GPU library.

What it computes (textbook definitions, written out plainly):

* ``ltlt`` -- Parlett & Reid's unblocked reduction of a skew-symmetric X to
  tridiagonal form with partial pivoting, P X P^T = L T L^T, in scalar C
  (``ltlt_oracle_body.h``): one column step at a time, pivot = first index of
  the largest magnitude, exchange, multipliers, skew rank-2 update of the
  trailing strict lower triangle.
* ``pfaffian`` -- Pf(X) = det(P) * prod_j T(2j, 2j+1), returned as
  (log|Pf|, sign), from Pf(B X B^T) = det(B) Pf(X).
* ``pfaffian_direct`` -- the same Pfaffian from the even column steps only
  (pivot, exchange, multipliers and rank-2 update at k = 0, 2, 4, ...; the
  odd columns are never eliminated because after step k row k has one
  nonzero entry and the Pfaffian expands along it).
* ``skew_update`` -- the definition of one trailing-matrix block update of
  the blocked method: new(i, c) = S(perm[i], perm[c]) + (Lx @ B^T)(i, c) on
  the strict lower triangle, with the mirrored upper entry, via one numpy
  matrix product.
* ``unpack`` -- reads L, the tridiagonal T and P back out of the packed
  output, for the residual P X P^T - L T L^T.
* ``solve`` / ``tridiag_skew_solve`` -- X^{-1} B from the factors:
  permutation, forward substitution with L, the two recurrences of the skew
  tridiagonal T, backward substitution with L^T, inverse permutation
  (triangular solves by scipy, the recurrences written out).
* complex skew-symmetric X (X^T = -X, complex128 / complex64): ``ltlt`` and
  ``pfaffian`` take the same steps in scalar C with the complex arithmetic
  written out (``ltlt_oracle_complex.h``): pivot by |re| + |im|, Smith's
  quotient; the Pfaffian comes back as (log|Pf|, phase Pf/|Pf|).

Every floating-point routine runs in the precision of its input (fp64, or fp32
for fp32 parity); the Pfaffian accumulates in fp64.

The convolution operator of the paper's section 3 (direct loops, im2col) has
its own module, ``oracle.conv``, with its own C source.

Pins (tests that tie these functions to facts outside themselves) live in
``tests/test_oracle_pins*.py``; no function here is unpinned.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ltlt_oracle.c")
_HDR = os.path.join(_HERE, "ltlt_oracle_body.h")
_HDR_C = os.path.join(_HERE, "ltlt_oracle_complex.h")
_LIB = os.path.join(_HERE, "libltlt_oracle.so")
_lock = threading.Lock()
_lib = None

GCC_FLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared", "-std=c99"]


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (no FMA contraction, no reassociation)."""
    stale = (not os.path.exists(_LIB)
             or os.path.getmtime(_LIB) < max(os.path.getmtime(_SRC), os.path.getmtime(_HDR),
                                             os.path.getmtime(_HDR_C)))
    if force or stale:
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *GCC_FLAGS, _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    from . import conv
    conv.build(force)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB):
                build()
            lib = ctypes.CDLL(_LIB)
            i64, p = ctypes.c_int64, ctypes.c_void_p
            for name in ("oracle_ltlt_f64", "oracle_ltlt_f32", "oracle_ltlt_c128", "oracle_ltlt_c64"):
                getattr(lib, name).argtypes = [i64, p, i64, p, i64]
                getattr(lib, name).restype = None
            for name in ("oracle_swap_f64", "oracle_swap_c128"):
                getattr(lib, name).argtypes = [i64, p, i64, i64, i64]
                getattr(lib, name).restype = None
            for name in ("oracle_pfaffian_f64", "oracle_pfaffian_f32", "oracle_pfaffian_c128",
                         "oracle_pfaffian_c64"):
                getattr(lib, name).argtypes = [i64, p, i64, p, p, p]
                getattr(lib, name).restype = None
            for name in ("oracle_pfaffian_direct_f64", "oracle_pfaffian_direct_f32"):
                getattr(lib, name).argtypes = [i64, p, i64, p, i64]
                getattr(lib, name).restype = None
            for name in ("oracle_ltlt_batched_f64", "oracle_ltlt_batched_f32"):
                getattr(lib, name).argtypes = [i64, i64, p, i64, i64, p, i64, p, p]
                getattr(lib, name).restype = None
            for name in ("oracle_ltlt_trace_f64", "oracle_ltlt_trace_f32"):
                getattr(lib, name).argtypes = [i64, p, i64, p, i64, p, p, p]
                getattr(lib, name).restype = None
            lib.oracle_set_threads.argtypes = [ctypes.c_int32]
            lib.oracle_set_threads.restype = None
            lib.oracle_get_threads.argtypes = []
            lib.oracle_get_threads.restype = ctypes.c_int32
            _lib = lib
    return _lib


def set_threads(t: int) -> None:
    """Threads for the real rank-2 update (OpenMP over its columns); the
    results are bitwise the same for any count."""
    _load().oracle_set_threads(int(t))


def get_threads() -> int:
    """Threads the real rank-2 update will use."""
    return int(_load().oracle_get_threads())


def _sfx(dtype) -> str:
    dt = np.dtype(dtype)
    if dt == np.float64:
        return "f64"
    if dt == np.float32:
        return "f32"
    if dt == np.complex128:
        return "c128"
    if dt == np.complex64:
        return "c64"
    raise TypeError("oracle supports float64, float32, complex128 and complex64 only")


def ltlt_colmajor(buf: np.ndarray, n: int, nsteps: int = -1):
    """Factor in place.  ``buf`` is a C-ordered (n, lda) array holding the
    column-major matrix (``buf[c, i]`` = element (i, c)); only its strict
    lower triangle (in column-major terms) is read or written.
    Returns the int32 pivot vector (0-based, LAPACK laswp order)."""
    lib = _load()
    if not (buf.flags.c_contiguous and buf.ndim == 2 and buf.shape[0] >= n):
        raise ValueError("buf must be a C-contiguous (n, lda) array")
    lda = buf.shape[1]
    ipiv = np.zeros(max(n, 1), dtype=np.int32)
    fn = getattr(lib, "oracle_ltlt_" + _sfx(buf.dtype))
    fn(n, buf.ctypes.data, lda, ipiv.ctypes.data, int(nsteps))
    return ipiv[:n]


def ltlt(X: np.ndarray, nsteps: int = -1):
    """Factor the skew matrix ``X`` (n x n, C order, X[i, j] = row i col j).

    Returns ``(packed, ipiv)`` where ``packed`` is an n x n array (row/col
    indexing) whose strict lower triangle holds alpha_k at (k+1, k) and
    L(r, k+1) at (r, k) for r >= k+2; its other entries are zero.
    """
    n = X.shape[0]
    buf = np.ascontiguousarray(X.T)          # column-major image of X
    ipiv = ltlt_colmajor(buf, n, nsteps)
    packed = np.tril(buf.T, -1)
    return np.ascontiguousarray(packed), ipiv


def ltlt_trace(X: np.ndarray, nsteps: int = -1):
    """``ltlt`` that also records each column step's pivot decision (real
    dtypes only).  Returns ``(packed, ipiv, best, runner, runner_mag)``:
    ``best[k]`` = |X(p_k, k)| at step k, ``runner[k]`` the first row of the
    largest magnitude among the other candidate rows (-1 if none) and
    ``runner_mag[k]`` its magnitude, in the input's precision."""
    lib = _load()
    n = X.shape[0]
    buf = np.ascontiguousarray(X.T)
    sfx = _sfx(buf.dtype)
    if sfx not in ("f64", "f32"):
        raise TypeError("ltlt_trace takes real matrices")
    ipiv = np.zeros(max(n, 1), dtype=np.int32)
    ns = max(n - 2, 1)
    best = np.zeros(ns, dtype=buf.dtype)
    runner = np.full(ns, -1, dtype=np.int32)
    rmag = np.zeros(ns, dtype=buf.dtype)
    getattr(lib, "oracle_ltlt_trace_" + sfx)(n, buf.ctypes.data, n, ipiv.ctypes.data, int(nsteps),
                                            best.ctypes.data, runner.ctypes.data, rmag.ctypes.data)
    packed = np.ascontiguousarray(np.tril(buf.T, -1))
    k = max(n - 2, 0)
    return packed, ipiv[:n], best[:k], runner[:k], rmag[:k]


def pfaffian_packed(packed: np.ndarray, ipiv: np.ndarray):
    """(log|Pf(X)|, sign) from the packed factors (row/col indexed n x n).
    Complex factors give (log|Pf(X)|, phase) with phase = Pf / |Pf| a Python
    complex (0 when Pf = 0)."""
    lib = _load()
    n = packed.shape[0]
    buf = np.ascontiguousarray(packed.T)     # column-major image
    logabs = ctypes.c_double(0.0)
    ip = np.ascontiguousarray(ipiv, dtype=np.int32)
    if np.iscomplexobj(packed):
        ph = np.zeros(2, dtype=np.float64)
        getattr(lib, "oracle_pfaffian_" + _sfx(packed.dtype))(n, buf.ctypes.data, n, ip.ctypes.data,
                                                              ctypes.byref(logabs), ph.ctypes.data)
        return float(logabs.value), complex(ph[0], ph[1])
    sign = ctypes.c_int32(0)
    fn = getattr(lib, "oracle_pfaffian_" + _sfx(packed.dtype))
    fn(n, buf.ctypes.data, n, ip.ctypes.data, ctypes.byref(logabs), ctypes.byref(sign))
    return float(logabs.value), int(sign.value)


def pfaffian(X: np.ndarray):
    """(log|Pf(X)|, sign) of a skew matrix via the factorization."""
    packed, ipiv = ltlt(X)
    return pfaffian_packed(packed, ipiv)


def pfaffian_direct(X: np.ndarray):
    """Pfaffian by the even column steps only (the odd columns are never
    eliminated: after step k, row k has the single entry T(k, k+1), and the
    Pfaffian expands along it).

    Returns ``(logabs, sign, alpha, ipiv)``: alpha[i] = alpha_{2i} of the even
    steps (n/2 values), ipiv the 0-based pivots with ipiv[k+1] = p_k for even
    k and ipiv[i] = i elsewhere.  Odd n gives (-inf, 0, [], identity)."""
    n = X.shape[0]
    buf = np.ascontiguousarray(X.T)          # column-major image of X
    ipiv = pfaffian_direct_colmajor(buf, n)
    out = np.tril(buf.T, -1)
    alpha = np.array([out[k + 1, k] for k in range(0, n - 1, 2)] if n % 2 == 0 else [], dtype=buf.dtype)
    logabs, sign = pfaffian_packed(np.ascontiguousarray(out), ipiv)
    return logabs, sign, alpha, ipiv


def pfaffian_direct_colmajor(buf: np.ndarray, n: int, nsteps: int = -1):
    """The even column steps in place on a C-ordered (n, lda) array holding
    the column-major matrix (as ``ltlt_colmajor``); ``nsteps >= 0`` stops
    after that many even steps.  Returns the int32 pivot vector."""
    lib = _load()
    if not (buf.flags.c_contiguous and buf.ndim == 2 and buf.shape[0] >= n):
        raise ValueError("buf must be a C-contiguous (n, lda) array")
    ipiv = np.zeros(max(n, 1), dtype=np.int32)
    getattr(lib, "oracle_pfaffian_direct_" + _sfx(buf.dtype))(n, buf.ctypes.data, buf.shape[1], ipiv.ctypes.data,
                                                               int(nsteps))
    return ipiv[:n]


def ltlt_batched(Xs: np.ndarray):
    """Factor a stack of skew matrices ``Xs`` (batch, n, n).

    Returns ``(packed, ipiv, logabs, sign)`` with packed (batch, n, n)."""
    lib = _load()
    batch, n, _ = Xs.shape
    buf = np.ascontiguousarray(np.transpose(Xs, (0, 2, 1)))
    ipiv = np.zeros((batch, max(n, 1)), dtype=np.int32)
    logabs = np.zeros(batch, dtype=np.float64)
    sign = np.zeros(batch, dtype=np.int32)
    fn = getattr(lib, "oracle_ltlt_batched_" + _sfx(Xs.dtype))
    fn(n, batch, buf.ctypes.data, n, n * n, ipiv.ctypes.data, ipiv.shape[1],
       logabs.ctypes.data, sign.ctypes.data)
    packed = np.tril(np.transpose(buf, (0, 2, 1)), -1)
    return np.ascontiguousarray(packed), ipiv[:, :n], logabs, sign


def swap_indices(X: np.ndarray, r: int, p: int) -> np.ndarray:
    """Q X Q^T for the transposition (r p), through the oracle's lower-storage
    exchange; returns the full skew matrix rebuilt from the strict lower part
    (fp64, or complex128 for complex X)."""
    lib = _load()
    n = X.shape[0]
    dt = np.complex128 if np.iscomplexobj(X) else np.float64
    buf = np.ascontiguousarray(X.T).astype(dt)
    getattr(lib, "oracle_swap_" + _sfx(dt))(n, buf.ctypes.data, n, r, p)
    low = np.tril(buf.T, -1)
    return low - low.T


def unpack(packed: np.ndarray, ipiv: np.ndarray):
    """Return (L, T, perm) with P X P^T = L T L^T, P[i, perm[i]] = 1.

    L is unit lower triangular with L[:, 0] = e_0 and L[r, k+1] = packed[r, k]
    (r >= k+2); T is skew tridiagonal with T[k+1, k] = packed[k+1, k];
    perm applies the exchanges (i, ipiv[i]) for i = 0 .. n-1 in order to the
    identity ordering, so (P X P^T)[i, j] = X[perm[i], perm[j]].
    """
    n = packed.shape[0]
    dt = np.complex128 if np.iscomplexobj(packed) else np.float64
    L = np.eye(n, dtype=dt)
    T = np.zeros((n, n), dtype=dt)
    for k in range(n - 1):
        T[k + 1, k] = packed[k + 1, k]
        T[k, k + 1] = -packed[k + 1, k]
    for k in range(max(n - 2, 0)):
        L[k + 2:, k + 1] = packed[k + 2:, k]
    perm = np.arange(n)
    for i in range(n):
        j = int(ipiv[i])
        perm[i], perm[j] = perm[j], perm[i]
    return L, T, perm


def tridiag_skew_solve(alpha: np.ndarray, R: np.ndarray) -> np.ndarray:
    """Solve T W = R for the skew tridiagonal T with T[k+1, k] = alpha[k],
    T[k, k+1] = -alpha[k] (n = len(alpha) + 1, n even), by its two
    recurrences: row 0 gives W[1] = -R[0] / alpha[0] and the even rows i give
    the odd unknowns forward, W[i+1] = (alpha[i-1] W[i-1] - R[i]) / alpha[i];
    row n-1 gives W[n-2] = R[n-1] / alpha[n-2] and the odd rows i give the
    even unknowns backward, W[i-1] = (R[i] + alpha[i] W[i+1]) / alpha[i-1].
    R is (n,) or (n, nrhs); fp64."""
    a = np.asarray(alpha, dtype=np.float64)
    R = np.asarray(R, dtype=np.float64)
    n = a.shape[0] + 1
    if n % 2:
        raise ValueError("a skew tridiagonal matrix of odd order is singular")
    W = np.zeros_like(R)
    W[1] = -R[0] / a[0]
    for i in range(2, n - 1, 2):
        W[i + 1] = (a[i - 1] * W[i - 1] - R[i]) / a[i]
    W[n - 2] = R[n - 1] / a[n - 2]
    for i in range(n - 3, 0, -2):
        W[i - 1] = (R[i] + a[i] * W[i + 1]) / a[i - 1]
    return W


def solve(packed: np.ndarray, ipiv: np.ndarray, B: np.ndarray) -> np.ndarray:
    """X^{-1} B from the factors (fp64).  With P X P^T = L T L^T (``unpack``),
    X x = b is L T L^T (P x) = P b, so: y = P b (y[i] = b[perm[i]]),
    z = L^{-1} y (unit lower, forward substitution), w = T^{-1} z (the two
    recurrences of ``tridiag_skew_solve``), u = L^{-T} w (backward
    substitution) and x = P^T u (x[perm[i]] = u[i]).  B is (n,) or
    (n, nrhs); n must be even (odd order: X is singular)."""
    from scipy.linalg import solve_triangular
    n = packed.shape[0]
    L, _, perm = unpack(np.asarray(packed, dtype=np.float64), ipiv)
    alpha = np.array([packed[k + 1, k] for k in range(n - 1)], dtype=np.float64)
    Bd = np.asarray(B, dtype=np.float64)
    y = Bd[perm]
    z = solve_triangular(L, y, lower=True, unit_diagonal=True)
    w = tridiag_skew_solve(alpha, z)
    u = solve_triangular(L.T, w, lower=False, unit_diagonal=True)
    x = np.empty_like(u)
    x[perm] = u
    return x


def residual(X: np.ndarray, packed: np.ndarray, ipiv: np.ndarray) -> float:
    """||P X P^T - L T L^T||_F / (n * eps * ||X||_F), eps of X's dtype."""
    n = X.shape[0]
    if n == 0:
        return 0.0
    wide = np.complex128 if np.iscomplexobj(X) else np.float64
    L, T, perm = unpack(packed.astype(wide), ipiv)
    Xd = X.astype(wide)
    PXP = Xd[np.ix_(perm, perm)]
    R = PXP - L @ T @ L.T
    eps = np.finfo(X.dtype).eps
    nx = np.linalg.norm(Xd)
    if nx == 0:
        return float(np.linalg.norm(R))
    return float(np.linalg.norm(R) / (n * eps * nx))


def skew_update(S: np.ndarray, Lx: np.ndarray, B: np.ndarray, perm: np.ndarray) -> np.ndarray:
    """One trailing-block update of the blocked method, by definition.

    ``S`` is the m x m skew matrix before the block (full storage), ``perm``
    maps each current index to the index it held before the block's exchanges,
    ``Lx`` and ``B`` are m x K.  Returns the full skew matrix whose strict
    lower entries are S[perm[i], perm[c]] + (Lx @ B.T)[i, c] (i > c) and whose
    upper entries are their negations, diagonal 0.
    """
    m = S.shape[0]
    P = S[np.ix_(perm, perm)]
    new = P + Lx @ B.T
    low = np.tril(new, -1)
    out = low - low.T
    assert out.shape == (m, m)
    return out
