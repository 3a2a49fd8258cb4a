"""CPU oracle for the convolution operator O = conv(F, I) (paper section 3).

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this module.  The GPU library never
links, imports or calls it, and it shares no code with the GPU library.

What it computes (``conv_oracle.c``, plain scalar C, written from the
definitions):

* ``out_size`` -- the output extent floor((h - k + 2p)/s) + 1 of section 3.
* ``conv_direct`` -- the direct seven-loop convolution of Figure 4, in fp64
  from fp32 inputs (each product exact, sums in the figure's loop order).
* ``conv_points`` -- single entries of O from the same sum, for sampled checks
  of problems too large for the full loops.
* ``im2col`` -- the explicit augmented matrix B^ of Figure 5 (K x N,
  K = kh kw ci rows, N = ho wo b columns).

Tensors are numpy arrays in Fortran order, so that memory holds them with the
leftmost index fastest, as section 3 stores them: I is (hi, wi, ci, b), F is
(kn, kh, kw, ci), O is (kn, ho, wo, b).  Padding p reads zeros outside the
input (see ``conv_oracle.c``).

Pins live in ``tests/test_oracle_pins_conv.py``: torch's CPU conv2d in fp64,
im2col followed by a numpy product, brute-force Python loops on tiny integer
cases, and closed forms (1 x 1 filters, shifted copies, all-ones counts), plus
the paper's Table 2 GEMM sizes and Table 1's im2col memory figure.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "conv_oracle.c")
_LIB = os.path.join(_HERE, "libconv_oracle.so")
_lock = threading.Lock()
_lib = None

GCC_FLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared", "-std=c99"]


def build(force: bool = False) -> str:
    stale = not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC)
    if force or stale:
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *GCC_FLAGS, _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build()
            lib = ctypes.CDLL(_LIB)
            i64, p = ctypes.c_int64, ctypes.c_void_p
            lib.oracle_conv_direct.argtypes = [i64] * 9 + [p, p, p]
            lib.oracle_conv_direct.restype = None
            lib.oracle_im2col.argtypes = [i64] * 8 + [p, p]
            lib.oracle_im2col.restype = None
            lib.oracle_conv_points.argtypes = [i64] * 9 + [p, p, i64, p, p]
            lib.oracle_conv_points.restype = None
            lib.oracle_conv_set_threads.argtypes = [ctypes.c_int32]
            lib.oracle_conv_set_threads.restype = None
            lib.oracle_conv_get_threads.argtypes = []
            lib.oracle_conv_get_threads.restype = ctypes.c_int32
            _lib = lib
    return _lib


def set_threads(t: int) -> None:
    """Threads over the batch loop; results are bitwise the same for any count."""
    _load().oracle_conv_set_threads(int(t))


def get_threads() -> int:
    return int(_load().oracle_conv_get_threads())


def out_size(h: int, k: int, s: int, p: int) -> int:
    """floor((h - k + 2p)/s) + 1 (section 3); the window must fit the padded input."""
    if s < 1 or p < 0 or k < 1 or h - k + 2 * p < 0:
        raise ValueError(f"no output: h={h} k={k} s={s} p={p}")
    return (h - k + 2 * p) // s + 1


def _f32(a, ndim, name):
    a = np.asarray(a)
    if a.dtype != np.float32 or a.ndim != ndim:
        raise TypeError(f"{name} must be a {ndim}-d float32 array")
    return np.asfortranarray(a)


def conv_direct(F, I, s: int = 1, p: int = 0) -> np.ndarray:
    """O = conv(F, I) by the direct loops of Figure 4, in fp64.
    F: (kn, kh, kw, ci) float32; I: (hi, wi, ci, b) float32; returns O as a
    Fortran-ordered (kn, ho, wo, b) float64 array."""
    F = _f32(F, 4, "F")
    I = _f32(I, 4, "I")
    kn, kh, kw, ci = F.shape
    hi, wi, ci2, b = I.shape
    if ci2 != ci:
        raise ValueError("F and I disagree on the channel count")
    ho, wo = out_size(hi, kh, s, p), out_size(wi, kw, s, p)
    O = np.zeros((kn, ho, wo, b), dtype=np.float64, order="F")
    _load().oracle_conv_direct(kn, kh, kw, ci, hi, wi, b, s, p, F.ctypes.data, I.ctypes.data, O.ctypes.data)
    return O


def conv_points(F, I, pts, s: int = 1, p: int = 0) -> np.ndarray:
    """Entries O[k, oh, ow, b] for the rows (k, oh, ow, b) of ``pts``, in fp64."""
    F = _f32(F, 4, "F")
    I = _f32(I, 4, "I")
    kn, kh, kw, ci = F.shape
    hi, wi, ci2, b = I.shape
    if ci2 != ci:
        raise ValueError("F and I disagree on the channel count")
    ho, wo = out_size(hi, kh, s, p), out_size(wi, kw, s, p)
    pts = np.ascontiguousarray(pts, dtype=np.int64).reshape(-1, 4)
    lim = np.array([kn, ho, wo, b])
    if ((pts < 0) | (pts >= lim)).any():
        raise ValueError("point outside O")
    out = np.empty(len(pts), dtype=np.float64)
    _load().oracle_conv_points(kn, kh, kw, ci, hi, wi, b, s, p, F.ctypes.data, I.ctypes.data,
                               len(pts), pts.ctypes.data, out.ctypes.data)
    return out


def im2col(I, kh: int, kw: int, s: int = 1, p: int = 0) -> np.ndarray:
    """The augmented matrix B^ of Figure 5: (kh kw ci) x (ho wo b), float32,
    Fortran-ordered."""
    I = _f32(I, 4, "I")
    hi, wi, ci, b = I.shape
    ho, wo = out_size(hi, kh, s, p), out_size(wi, kw, s, p)
    B = np.empty((kh * kw * ci, ho * wo * b), dtype=np.float32, order="F")
    _load().oracle_im2col(kh, kw, ci, hi, wi, b, s, p, I.ctypes.data, B.ctypes.data)
    return B


def conv_abs(F, I, s: int = 1, p: int = 0) -> np.ndarray:
    """conv(|F|, |I|): the sum of the magnitudes of the terms of each output,
    the scale of the rounding-error bound of any fp32 evaluation order."""
    return conv_direct(np.abs(F), np.abs(I), s, p)
