"""Seeded synthetic tensors for the convolution operator, and the layer shapes.

Like the rest of ``synth`` this module only draws random numbers and lays them
out; it computes no part of a convolution.  Tensors come back as float32
numpy arrays in Fortran order, so memory holds them with the leftmost index
fastest, the storage convention of the paper's section 3:

* input  I: (hi, wi, ci, b)
* filters F: (kn, kh, kw, ci)

``ALEXNET_CONV`` lists the convolution layers of the AlexNet model as the
paper's Table 2 gives them (input hi x wi x ci, filters kn x kh x kw x ci).
The table does not print stride or padding; the values here (stride 4 for
the first layer, 1 for the others, no padding) are the ones that reproduce
the table's GEMM column counts (2916 b, 2601 b, 625 b, 121 b) through the
output-size formula of section 3.  The fifth layer's row prints 384 filters
in its kernel column but m = 256 in its GEMM column; the GEMM column is taken
(256 filters).

Value recipe (inference): inputs are activations after a ReLU-like
nonlinearity, uniform on [0, 1); filters are He-style Gaussians with variance
2 / (kh kw ci).  ``int_tensor`` draws small integers instead, for cases where
every fp32 sum is exact.
"""
from __future__ import annotations

import numpy as np

from . import rng_for

ALEXNET_CONV = [
    # name, hi, wi, ci, kn, kh, kw, stride, pad
    dict(layer=2, hi=224, wi=224, ci=3, kn=64, kh=11, kw=11, s=4, p=0),
    dict(layer=4, hi=55, wi=55, ci=64, kn=192, kh=5, kw=5, s=1, p=0),
    dict(layer=6, hi=27, wi=27, ci=192, kn=384, kh=3, kw=3, s=1, p=0),
    dict(layer=7, hi=13, wi=13, ci=384, kn=384, kh=3, kw=3, s=1, p=0),
    dict(layer=8, hi=13, wi=13, ci=384, kn=256, kh=3, kw=3, s=1, p=0),
]


# The benchmarked batch: the largest batch size of the paper's AlexNet runs
# (section 5.4 runs b up to 80).
ALEXNET_BATCH = 80


def layer_seed(spec: dict) -> int:
    """Seed of one layer's synthetic tensors in the benchmarked workload."""
    return 1000 + int(spec["layer"])


def _fortran(flat: np.ndarray, shape) -> np.ndarray:
    return np.asfortranarray(flat.reshape(shape, order="F"))


def input_tensor(hi: int, wi: int, ci: int, b: int, seed: int) -> np.ndarray:
    """I (hi, wi, ci, b), uniform on [0, 1), float32; memory order = draw order."""
    rng = rng_for(seed, 0)
    return _fortran(rng.random(hi * wi * ci * b, dtype=np.float32), (hi, wi, ci, b))


def filter_tensor(kn: int, kh: int, kw: int, ci: int, seed: int) -> np.ndarray:
    """F (kn, kh, kw, ci), N(0, 2/(kh kw ci)), float32."""
    rng = rng_for(seed, 1)
    g = rng.standard_normal(kn * kh * kw * ci) * np.sqrt(2.0 / (kh * kw * ci))
    return _fortran(g.astype(np.float32), (kn, kh, kw, ci))


def int_tensor(shape, seed: int, lo: int = -4, hi: int = 4, index: int = 2) -> np.ndarray:
    """Integers uniform on [lo, hi] stored as float32, Fortran order."""
    rng = rng_for(seed, index)
    n = int(np.prod(shape))
    return _fortran(rng.integers(lo, hi + 1, size=n).astype(np.float32), tuple(shape))


def layer_tensors(spec: dict, b: int, seed: int):
    """(F, I) for one layer of ``ALEXNET_CONV`` (or any dict with the same
    keys) at batch size b."""
    F = filter_tensor(spec["kn"], spec["kh"], spec["kw"], spec["ci"], seed)
    I = input_tensor(spec["hi"], spec["wi"], spec["ci"], b, seed)
    return F, I
