"""Test-side helpers for the convolution: moving tensors stored leftmost index
fastest (numpy Fortran order) to and from the GPU, and the comparison rule.

Comparison rule (fp32 CONVGEMM against the fp64 oracle):
* integer-valued inputs whose every partial sum is an integer below 2^24 are
  summed exactly in fp32 in any order: the results must be bit-identical;
* otherwise every entry must satisfy |O - O_ref| <= gamma_K * conv(|F|, |I|)
  + tiny, gamma_K = K u / (1 - K u), u = 2^-24, K = kh kw ci: the worst-case
  bound of any fp32 evaluation order of a K-term sum of exact products (fp32
  products of fp32 inputs round once more: K+1 roundings, covered by using
  K + 1), and the normwise error max|O - O_ref| / max|O_ref| must stay below
  1e-5.
"""
from __future__ import annotations

import numpy as np
import torch

U32 = 2.0 ** -24


def dev(a: np.ndarray) -> torch.Tensor:
    """numpy array (any order) -> GPU tensor of the same shape stored
    leftmost index fastest."""
    a = np.asfortranarray(a)
    shape = a.shape
    strides, acc = [], 1
    for d in shape:
        strides.append(acc)
        acc *= d
    flat = torch.from_numpy(np.ravel(a, order="F").copy()).cuda()
    return flat.as_strided(shape, tuple(strides))


def host(t: torch.Tensor) -> np.ndarray:
    """GPU tensor stored leftmost index fastest -> numpy Fortran array."""
    flat = t.as_strided((t.numel(),), (1,)).cpu().numpy()
    return np.asfortranarray(flat.reshape(tuple(t.shape), order="F"))


def bound(F, I, s, p, oracle_conv):
    K = F.shape[1] * F.shape[2] * F.shape[3]
    g = (K + 1) * U32 / (1 - (K + 1) * U32)
    return g * oracle_conv.conv_abs(F, I, s, p) + 1e-30


def check_close(got, ref, bnd, what=""):
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got.astype(np.float64) - ref)
    worst = np.unravel_index(np.argmax(err - bnd), err.shape)
    assert (err <= bnd).all(), f"{what}: error {err[worst]:.3e} > bound {bnd[worst]:.3e} at {worst}"
    nw = err.max() / max(np.abs(ref).max(), 1e-30)
    assert nw <= 1e-5, f"{what}: normwise error {nw:.3e}"
    return nw
