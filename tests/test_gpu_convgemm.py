"""GPU parity of CONVGEMM (``convgemm_f32`` through the C ABI) against the
convolution oracle (direct loops of the paper's Figure 4, fp64).

* integer-valued inputs: bit-exact (every partial sum is an integer < 2^24);
* Gaussian / uniform inputs: within gamma_{K+1} * conv(|F|, |I|) entrywise and
  1e-5 normwise (see ``conv_util``);
* both kernels: the LDS-staged gather (path 1) in every workgroup tile (64x64,
  64x128, 64x256, 128x128, 192x128) and the register-direct one (path 2, no
  padding) in every tile (64x64, 64x128, 128x64, 128x128), on the same
  ragged problem (filter count, contraction length and output count not
  multiples of any tile), both with few tiles (32-row contraction chunks) and
  with many (16-row chunks), with and without padding; strides 1-4, padding
  0-3, non-square inputs and filters, 1x1 filters, a single output position, an empty batch, kn not a
  multiple of 4 and a misaligned output (scalar epilogue), accumulate mode;
* short grids with long contractions, whose tiles' contractions the
  automatic choice splits over several workgroups (atomic adds), exact and
  accumulating;
* the AlexNet layers of the paper's Table 2 at b = 2 in full, and at the
  benchmarked b = 80 on sampled outputs (each computed one by one by the
  oracle) plus bit-exact integer runs sampled the same way.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2005_06410_amd as lt
import synth
from conv_util import bound, check_close, dev, host
from oracle import conv as oc
from synth import conv as sc

pytestmark = pytest.mark.gpu

TILES = [(64, 64), (64, 128), (64, 256), (128, 128), (192, 128)]
DIRECT_TILES = [(64, 64), (64, 128), (128, 64), (128, 128)]


def run(F, I, s, p, tile=(0, 0), out=None, accumulate=False, path=None):
    Fd, Id = dev(F), dev(I)
    if path is None:
        path = 0 if tile == (0, 0) else 1
    O = lt.convgemm(Fd, Id, stride=s, pad=p, tile=tile, out=out, accumulate=accumulate, path=path)
    torch.cuda.synchronize()
    return O


def int_case(kn, kh, kw, ci, hi, wi, b, seed, lo=-3, hi_=3):
    F = sc.int_tensor((kn, kh, kw, ci), seed, lo, hi_, index=5)
    I = sc.int_tensor((hi, wi, ci, b), seed, lo, hi_, index=6)
    return F, I


def gauss_case(kn, kh, kw, ci, hi, wi, b, seed):
    return sc.filter_tensor(kn, kh, kw, ci, seed), sc.input_tensor(hi, wi, ci, b, seed)


RAGGED = (70, 3, 3, 7, 23, 17, 3)     # kn=70, K=63, N=21*15*3=945 at s=1 p=0


@pytest.mark.parametrize("tile", TILES)
def test_every_tile_integer_exact(tile):
    kn, kh, kw, ci, hi, wi, b = RAGGED
    F, I = int_case(kn, kh, kw, ci, hi, wi, b, 40)
    print(f"[conv] tile {tile} integer ragged", flush=True)
    got = host(run(F, I, 1, 0, tile))
    assert np.array_equal(got.astype(np.float64), oc.conv_direct(F, I, 1, 0))


@pytest.mark.parametrize("tile", TILES)
def test_every_tile_gaussian(tile):
    kn, kh, kw, ci, hi, wi, b = RAGGED
    F, I = gauss_case(kn, kh, kw, ci, hi, wi, b, 41)
    print(f"[conv] tile {tile} gaussian ragged, stride 2 pad 1", flush=True)
    got = host(run(F, I, 2, 1, tile))
    check_close(got, oc.conv_direct(F, I, 2, 1), bound(F, I, 2, 1, oc), f"tile {tile}")


# kn=70, K=63, N = 58*58*40 = 134560 (stride 1, no padding) or 60*60*40 with
# padding 1: at least 1052 tiles for every tile shape, so the 16-row chunk
# kernels run.
LONG = (70, 3, 3, 7, 60, 60, 40)


@pytest.mark.parametrize("tile", TILES)
def test_every_tile_many_tiles_integer_exact(tile):
    kn, kh, kw, ci, hi, wi, b = LONG
    F, I = int_case(kn, kh, kw, ci, hi, wi, b, 50)
    print(f"[conv] tile {tile} integer, many tiles", flush=True)
    got = host(run(F, I, 1, 0, tile))
    assert np.array_equal(got.astype(np.float64), oc.conv_direct(F, I, 1, 0))


@pytest.mark.parametrize("tile", TILES)
def test_every_tile_many_tiles_padded_gaussian(tile):
    kn, kh, kw, ci, hi, wi, b = LONG
    F, I = gauss_case(kn, kh, kw, ci, hi, wi, b, 51)
    print(f"[conv] tile {tile} gaussian, many tiles, pad 1", flush=True)
    got = host(run(F, I, 1, 1, tile))
    check_close(got, oc.conv_direct(F, I, 1, 1), bound(F, I, 1, 1, oc), f"tile {tile} padded")


@pytest.mark.parametrize("tile", DIRECT_TILES)
@pytest.mark.parametrize("shape", ["ragged", "long"])
def test_direct_every_tile_integer_exact(tile, shape):
    kn, kh, kw, ci, hi, wi, b = RAGGED if shape == "ragged" else LONG
    F, I = int_case(kn, kh, kw, ci, hi, wi, b, 52)
    print(f"[conv] register-direct tile {tile} integer {shape}", flush=True)
    got = host(run(F, I, 1, 0, tile, path=2))
    assert np.array_equal(got.astype(np.float64), oc.conv_direct(F, I, 1, 0))


@pytest.mark.parametrize("tile", DIRECT_TILES)
def test_direct_every_tile_gaussian_strided(tile):
    kn, kh, kw, ci, hi, wi, b = RAGGED
    F, I = gauss_case(kn, kh, kw, ci, hi, wi, b, 53)
    print(f"[conv] register-direct tile {tile} gaussian stride 2", flush=True)
    got = host(run(F, I, 2, 0, tile, path=2))
    check_close(got, oc.conv_direct(F, I, 2, 0), bound(F, I, 2, 0, oc), f"direct tile {tile}")


GEOMS = [
    # kn, kh, kw, ci, hi, wi, b, s, p
    (5, 3, 2, 3, 11, 9, 3, 2, 1),
    (16, 1, 1, 9, 7, 5, 4, 1, 0),       # 1x1 filters: a channel product
    (12, 4, 4, 2, 9, 13, 2, 3, 2),
    (8, 5, 3, 4, 10, 12, 2, 4, 3),      # stride above the filter: skipped rows
    (7, 3, 3, 5, 3, 3, 1, 1, 0),        # one output position (kn not a multiple of 4)
    (3, 2, 2, 1, 4, 4, 1, 2, 3),        # padding wider than the filter: zero borders
    (33, 7, 7, 3, 30, 28, 2, 2, 3),
    (130, 3, 3, 17, 12, 12, 5, 1, 1),
    (9, 4, 3, 3, 17, 14, 2, 3, 0),
    (66, 5, 5, 6, 20, 19, 3, 2, 0),
]


@pytest.mark.parametrize("g", GEOMS)
def test_geometries_integer_exact(g):
    kn, kh, kw, ci, hi, wi, b, s, p = g
    F, I = int_case(kn, kh, kw, ci, hi, wi, b, 42)
    print(f"[conv] geometry {g} integer", flush=True)
    got = host(run(F, I, s, p))
    assert np.array_equal(got.astype(np.float64), oc.conv_direct(F, I, s, p))


@pytest.mark.parametrize("g", [g for g in GEOMS if g[8] == 0])
@pytest.mark.parametrize("path", [1, 2])
def test_unpadded_geometries_both_paths_integer_exact(g, path):
    kn, kh, kw, ci, hi, wi, b, s, p = g
    F, I = int_case(kn, kh, kw, ci, hi, wi, b, 54)
    print(f"[conv] geometry {g} path {path} integer", flush=True)
    got = host(run(F, I, s, p, path=path))
    assert np.array_equal(got.astype(np.float64), oc.conv_direct(F, I, s, p))


@pytest.mark.parametrize("g", GEOMS)
def test_geometries_gaussian(g):
    kn, kh, kw, ci, hi, wi, b, s, p = g
    F, I = gauss_case(kn, kh, kw, ci, hi, wi, b, 43)
    print(f"[conv] geometry {g} gaussian", flush=True)
    got = host(run(F, I, s, p))
    check_close(got, oc.conv_direct(F, I, s, p), bound(F, I, s, p, oc), str(g))


@pytest.mark.parametrize("path", [1, 2])
def test_accumulate_adds_to_output(path):
    kn, kh, kw, ci, hi, wi, b = RAGGED
    F, I = gauss_case(kn, kh, kw, ci, hi, wi, b, 44)
    ho, wo = hi - kh + 1, wi - kw + 1
    O0 = np.asfortranarray(synth.rng_for(45).standard_normal((kn, ho, wo, b)).astype(np.float32))
    out = dev(O0)
    got = host(run(F, I, 1, 0, out=out, accumulate=True, path=path))
    ref = oc.conv_direct(F, I, 1, 0) + O0.astype(np.float64)
    bnd = bound(F, I, 1, 0, oc) + U_ROUND * (np.abs(ref) + np.abs(O0))
    check_close(got, ref, bnd, "accumulate")


U_ROUND = 2.0 ** -24


@pytest.mark.parametrize("path", [1, 2])
def test_misaligned_output_uses_scalar_stores(path):
    kn, kh, kw, ci, hi, wi, b = 8, 3, 3, 4, 10, 9, 2
    F, I = int_case(kn, kh, kw, ci, hi, wi, b, 46)
    ho, wo = hi - kh + 1, wi - kw + 1
    n = kn * ho * wo * b
    flat = torch.full((n + 1,), 7.0, dtype=torch.float32, device="cuda")
    out = flat[1:].as_strided((kn, ho, wo, b), (1, kn, kn * ho, kn * ho * wo))
    assert out.data_ptr() % 16 != 0
    got = host(run(F, I, 1, 0, out=out, path=path))
    assert np.array_equal(got.astype(np.float64), oc.conv_direct(F, I, 1, 0))
    assert float(flat[0].item()) == 7.0


@pytest.mark.parametrize("path", [1, 2])
@pytest.mark.parametrize("kn,kh,kw,ci", [(1, 1, 1, 1), (3, 1, 1, 15), (5, 2, 2, 4), (4, 1, 1, 17),
                                         (2, 31, 1, 1), (6, 3, 11, 1)])
def test_short_contractions_integer_exact(path, kn, kh, kw, ci):
    """K = 1, 15, 16, 17, 31, 33: a single partial group, exact multiples of
    the 16-row group, and one row past it; kn = 1 (one filter)."""
    hi, wi, b = kh + 4, kw + 3, 2
    F, I = int_case(kn, kh, kw, ci, hi, wi, b, 55)
    print(f"[conv] short contraction K={kh * kw * ci} kn={kn} path {path}", flush=True)
    got = host(run(F, I, 1, 0, path=path))
    assert np.array_equal(got.astype(np.float64), oc.conv_direct(F, I, 1, 0))


# Short grid, long contraction: the automatic register-direct choice (64 x 64
# tiles, fewer than three per CU) splits each tile's contraction over two or
# four workgroups that add into O atomically (O cleared first unless
# accumulating).  K = 3*3*300 = 2700 (169 groups of 16: two parts), and
# 3*3*600 = 5400 (338 groups: four parts); kn = 70 is not a multiple of 4.
SPLITS = [(70, 3, 3, 300, 9, 8, 2), (36, 3, 3, 600, 7, 9, 3)]


@pytest.mark.parametrize("g", SPLITS)
def test_split_contraction_integer_exact(g):
    kn, kh, kw, ci, hi, wi, b = g
    F, I = int_case(kn, kh, kw, ci, hi, wi, b, 57, -2, 2)
    ho, wo = hi - kh + 1, wi - kw + 1
    print(f"[conv] split contraction K={kh * kw * ci} kn={kn} N={ho * wo * b}", flush=True)
    # a stale output must not leak into the result
    out = dev(np.asfortranarray(np.full((kn, ho, wo, b), 9.0, dtype=np.float32)))
    got = host(run(F, I, 1, 0, out=out))
    assert np.array_equal(got.astype(np.float64), oc.conv_direct(F, I, 1, 0))
    # accumulate: O += conv(F, I), exact for integers
    O0 = sc.int_tensor((kn, ho, wo, b), 58, -5, 5, index=7)
    got = host(run(F, I, 1, 0, out=dev(O0), accumulate=True))
    assert np.array_equal(got.astype(np.float64), oc.conv_direct(F, I, 1, 0) + O0.astype(np.float64))


@pytest.mark.parametrize("g", SPLITS)
def test_split_contraction_gaussian(g):
    kn, kh, kw, ci, hi, wi, b = g
    F, I = gauss_case(kn, kh, kw, ci, hi, wi, b, 59)
    got = host(run(F, I, 1, 0))
    check_close(got, oc.conv_direct(F, I, 1, 0), bound(F, I, 1, 0, oc), f"split {g}")


def test_long_contraction_falls_back_to_lds_staging():
    """K = 3*3*2000 = 18000 rows exceeds the register-direct kernel's row table:
    the automatic choice takes the LDS-staged kernel."""
    kn, kh, kw, ci, hi, wi, b = 8, 3, 3, 2000, 5, 6, 2
    F, I = int_case(kn, kh, kw, ci, hi, wi, b, 56, -2, 2)
    print("[conv] long contraction K=18000", flush=True)
    got = host(run(F, I, 1, 0))
    assert np.array_equal(got.astype(np.float64), oc.conv_direct(F, I, 1, 0))


def test_empty_batch():
    F = dev(sc.filter_tensor(4, 3, 3, 2, 1))
    I = torch.empty(0, dtype=torch.float32, device="cuda").as_strided((6, 6, 2, 0), (1, 6, 36, 72))
    O = lt.convgemm(F, I)
    torch.cuda.synchronize()
    assert tuple(O.shape) == (4, 4, 4, 0)


@pytest.mark.parametrize("spec", sc.ALEXNET_CONV, ids=lambda s: f"layer{s['layer']}")
def test_alexnet_layer_b2_full(spec):
    """Every output of an AlexNet layer (Table 2 shapes) at b = 2."""
    F, I = sc.layer_tensors(spec, 2, sc.layer_seed(spec))
    print(f"[conv] AlexNet layer {spec['layer']} b=2", flush=True)
    got = host(run(F, I, spec["s"], spec["p"]))
    ref = oc.conv_direct(F, I, spec["s"], spec["p"])
    check_close(got, ref, bound(F, I, spec["s"], spec["p"], oc), f"layer {spec['layer']}")


def sample_points(shape, count, seed):
    """Random output positions plus every corner and the first/last entries
    along each dimension (tile edges in both GEMM directions)."""
    rng = synth.rng_for(seed)
    pts = np.stack([rng.integers(0, d, count) for d in shape], axis=1)
    edges = []
    for k in (0, 1, 63, 64, 127, 128, 191, 192, shape[0] - 1):
        for b in (0, shape[3] - 1):
            for oh in (0, shape[1] - 1):
                for ow in (0, shape[2] - 1):
                    if k < shape[0]:
                        edges.append((k, oh, ow, b))
    return np.concatenate([pts, np.array(edges, dtype=np.int64)])


@pytest.mark.parametrize("spec", sc.ALEXNET_CONV, ids=lambda s: f"layer{s['layer']}")
def test_alexnet_layer_full_batch_sampled(spec):
    """The benchmarked configuration (b = 80, automatic tile, the benchmark's
    inputs): 20000 sampled outputs against the oracle's one-by-one sums, and
    the output checked finite everywhere."""
    b = sc.ALEXNET_BATCH
    F, I = sc.layer_tensors(spec, b, sc.layer_seed(spec))
    print(f"[conv] AlexNet layer {spec['layer']} b={b} sampled", flush=True)
    O = run(F, I, spec["s"], spec["p"])
    assert bool(torch.isfinite(O).all())
    pts = sample_points(tuple(O.shape), 20000, 47 + spec["layer"])
    idx = torch.from_numpy(pts).cuda()
    got = O[idx[:, 0], idx[:, 1], idx[:, 2], idx[:, 3]].double().cpu().numpy()
    ref = oc.conv_points(F, I, pts, spec["s"], spec["p"])
    absref = oc.conv_points(np.abs(F), np.abs(I), pts, spec["s"], spec["p"])
    K = spec["kh"] * spec["kw"] * spec["ci"]
    g = (K + 1) * U_ROUND / (1 - (K + 1) * U_ROUND)
    err = np.abs(got - ref)
    assert (err <= g * absref).all(), f"max error {err.max():.3e}"
    assert err.max() / np.abs(ref).max() <= 1e-5


@pytest.mark.parametrize("spec", sc.ALEXNET_CONV, ids=lambda s: f"layer{s['layer']}")
def test_alexnet_layer_full_batch_integer_sampled(spec):
    """Integer-valued inputs at the benchmarked size: sampled outputs bit-exact."""
    b = sc.ALEXNET_BATCH
    F = sc.int_tensor((spec["kn"], spec["kh"], spec["kw"], spec["ci"]), 48, -3, 3, index=7)
    I = sc.int_tensor((spec["hi"], spec["wi"], spec["ci"], b), 48, 0, 3, index=8)
    print(f"[conv] AlexNet layer {spec['layer']} b={b} integer sampled", flush=True)
    O = run(F, I, spec["s"], spec["p"])
    pts = sample_points(tuple(O.shape), 20000, 49 + spec["layer"])
    idx = torch.from_numpy(pts).cuda()
    got = O[idx[:, 0], idx[:, 1], idx[:, 2], idx[:, 3]].double().cpu().numpy()
    assert np.array_equal(got, oc.conv_points(F, I, pts, spec["s"], spec["p"]))
