"""Pins of the convolution oracle (``oracle.conv``) to facts outside itself.

* the paper's Table 2: GEMM sizes m x n x k of every AlexNet layer from the
  output-size formula, and Table 1's 15.87 MiB per batch element for the
  largest explicit im2col matrix of AlexNet;
* torch's CPU conv2d in fp64 (a library routine for the same operator);
* im2col (Figure 5) followed by a numpy matrix product equals the direct
  loops (the identity conv(F, I) = F^ . im2col(I) of section 4);
* brute-force Python loops on tiny integer cases, bit-exact;
* closed forms: 1 x 1 filters are a plain matrix product over channels, a
  one-hot filter copies a shifted input channel, all-ones inputs count the
  window taps that fall inside the padded input;
* the output-size formula against a count of window positions.

The cases use non-square inputs and filters, strides 1-3, padding 0-2, and
several channels and batch entries, so that an exchanged index, a wrong stride
or padding sign, or a dropped term changes some output.
"""
from __future__ import annotations

import os

import numpy as np
import pytest
import torch

import synth
from oracle import conv as oc
from synth import conv as sc

HERE = os.path.dirname(os.path.abspath(__file__))

CASES = [
    # kn, kh, kw, ci, hi, wi, b, s, p
    (3, 3, 3, 2, 7, 6, 2, 1, 0),
    (5, 2, 3, 3, 9, 8, 3, 2, 1),
    (4, 3, 2, 2, 11, 7, 2, 3, 2),
    (2, 1, 1, 4, 5, 6, 2, 1, 0),
    (6, 5, 4, 1, 10, 12, 1, 2, 0),
    (3, 4, 4, 3, 8, 8, 2, 1, 2),
]


def tensors(case, seed, integer=False):
    kn, kh, kw, ci, hi, wi, b, s, p = case
    if integer:
        F = sc.int_tensor((kn, kh, kw, ci), seed, index=3)
        I = sc.int_tensor((hi, wi, ci, b), seed, index=4)
    else:
        F = sc.filter_tensor(kn, kh, kw, ci, seed)
        I = sc.input_tensor(hi, wi, ci, b, seed) - np.float32(0.5)
        I = np.asfortranarray(I.astype(np.float32))
    return F, I


def brute_force(F, I, s, p):
    kn, kh, kw, ci = F.shape
    hi, wi, _, b = I.shape
    ho = (hi - kh + 2 * p) // s + 1
    wo = (wi - kw + 2 * p) // s + 1
    O = np.zeros((kn, ho, wo, b))
    for k in range(kn):
        for oh in range(ho):
            for ow in range(wo):
                for bb in range(b):
                    t = 0.0
                    for c in range(ci):
                        for y in range(kh):
                            for x in range(kw):
                                hh, ww = s * oh + y - p, s * ow + x - p
                                if 0 <= hh < hi and 0 <= ww < wi:
                                    t += float(F[k, y, x, c]) * float(I[hh, ww, c, bb])
                    O[k, oh, ow, bb] = t
    return O


def read_table(name):
    rows = []
    for line in open(os.path.join(HERE, "golden", name)):
        line = line.split("#")[0].split()
        if line:
            rows.append(line)
    return rows


def test_table2_gemm_sizes():
    rows = read_table("alexnet_conv_table2.txt")
    assert len(rows) == len(sc.ALEXNET_CONV) == 5
    for row, spec in zip(rows, sc.ALEXNET_CONV):
        layer, hi, wi, ci, kn, kh, kw, m, n_per_b, k = map(int, row)
        assert (layer, hi, wi, ci, kh, kw) == (spec["layer"], spec["hi"], spec["wi"], spec["ci"],
                                               spec["kh"], spec["kw"])
        # m is the filter count (the last row's kernel column prints 384, its m 256)
        assert spec["kn"] == m
        assert kn == m or layer == 8
        ho = oc.out_size(hi, kh, spec["s"], spec["p"])
        wo = oc.out_size(wi, kw, spec["s"], spec["p"])
        assert ho * wo == n_per_b
        assert kh * kw * ci == k


def test_table1_alexnet_im2col_memory():
    (model, mib), = read_table("cnn_im2col_memory_table1.txt")
    assert model == "AlexNet"
    sizes = []
    for spec in sc.ALEXNET_CONV:
        ho = oc.out_size(spec["hi"], spec["kh"], spec["s"], spec["p"])
        wo = oc.out_size(spec["wi"], spec["kw"], spec["s"], spec["p"])
        sizes.append(spec["kh"] * spec["kw"] * spec["ci"] * ho * wo * 4)
    # the table prints the figure as approximately 15.87 (16646400 B = 15.875 MiB)
    assert abs(max(sizes) / 2 ** 20 - float(mib)) < 0.01
    # and the oracle's im2col of that layer at b = 1 has exactly that size
    spec = sc.ALEXNET_CONV[int(np.argmax(sizes))]
    I = sc.input_tensor(spec["hi"], spec["wi"], spec["ci"], 1, 9)
    B = oc.im2col(I, spec["kh"], spec["kw"], spec["s"], spec["p"])
    assert B.nbytes == max(sizes)


def test_out_size_counts_window_positions():
    for h in range(1, 14):
        for k in range(1, 6):
            for s in range(1, 4):
                for p in range(0, 3):
                    if h - k + 2 * p < 0:
                        with pytest.raises(ValueError):
                            oc.out_size(h, k, s, p)
                        continue
                    # window starts -p, -p+s, ... whose last tap stays inside h + p
                    count = sum(1 for st in range(-p, h + p) if (st + p) % s == 0 and st + k - 1 <= h + p - 1)
                    assert oc.out_size(h, k, s, p) == count


@pytest.mark.parametrize("case", CASES)
def test_direct_matches_torch_conv2d(case):
    kn, kh, kw, ci, hi, wi, b, s, p = case
    F, I = tensors(case, 11)
    O = oc.conv_direct(F, I, s, p)
    x = torch.from_numpy(np.ascontiguousarray(I.transpose(3, 2, 0, 1))).double()
    w = torch.from_numpy(np.ascontiguousarray(F.transpose(0, 3, 1, 2))).double()
    y = torch.nn.functional.conv2d(x, w, stride=s, padding=p)
    ref = y.permute(1, 2, 3, 0).numpy()
    assert O.shape == ref.shape
    assert np.abs(O - ref).max() <= 1e-12 * max(1.0, np.abs(ref).max())


@pytest.mark.parametrize("case", CASES)
def test_brute_force_integers_exact(case):
    kn, kh, kw, ci, hi, wi, b, s, p = case
    F, I = tensors(case, 12, integer=True)
    assert np.array_equal(oc.conv_direct(F, I, s, p), brute_force(F, I, s, p))


@pytest.mark.parametrize("case", CASES)
def test_im2col_times_filters_equals_direct(case):
    kn, kh, kw, ci, hi, wi, b, s, p = case
    F, I = tensors(case, 13)
    B = oc.im2col(I, kh, kw, s, p)
    A = F.reshape(kn, kh * kw * ci, order="F").astype(np.float64)
    C = A @ B.astype(np.float64)
    ho, wo = oc.out_size(hi, kh, s, p), oc.out_size(wi, kw, s, p)
    O = oc.conv_direct(F, I, s, p)
    assert np.abs(C.reshape(kn, ho, wo, b, order="F") - O).max() <= 1e-12 * max(1.0, np.abs(O).max())


def test_im2col_brute_force():
    case = CASES[2]
    kn, kh, kw, ci, hi, wi, b, s, p = case
    _, I = tensors(case, 14)
    B = oc.im2col(I, kh, kw, s, p)
    ho, wo = oc.out_size(hi, kh, s, p), oc.out_size(wi, kw, s, p)
    ref = np.zeros((kh * kw * ci, ho * wo * b), dtype=np.float32)
    for bb in range(b):
        for ow in range(wo):
            for oh in range(ho):
                col = oh + ow * ho + bb * ho * wo
                for c in range(ci):
                    for x in range(kw):
                        for y in range(kh):
                            hh, ww = s * oh + y - p, s * ow + x - p
                            if 0 <= hh < hi and 0 <= ww < wi:
                                ref[y + x * kh + c * kh * kw, col] = I[hh, ww, c, bb]
    assert np.array_equal(B, ref)


def test_one_by_one_filter_is_channel_product():
    kn, ci, hi, wi, b = 5, 7, 6, 4, 3
    F = sc.filter_tensor(kn, 1, 1, ci, 15)
    I = sc.input_tensor(hi, wi, ci, b, 15)
    O = oc.conv_direct(F, I, 1, 0)
    A = F[:, 0, 0, :].astype(np.float64)                          # kn x ci
    X = I.astype(np.float64).transpose(2, 0, 1, 3).reshape(ci, -1)  # ci x (hi wi b)
    ref = (A @ X).reshape(kn, hi, wi, b)
    assert np.abs(O - ref).max() <= 1e-12


@pytest.mark.parametrize("case", CASES)
def test_one_hot_filter_copies_shifted_channel(case):
    kn, kh, kw, ci, hi, wi, b, s, p = case
    _, I = tensors(case, 16)
    y0, x0 = kh - 1, kw // 2
    F = np.zeros((kn, kh, kw, ci), dtype=np.float32, order="F")
    for k in range(kn):
        F[k, y0, x0, k % ci] = 1.0
    O = oc.conv_direct(F, I, s, p)
    ho, wo = O.shape[1], O.shape[2]
    for k in range(kn):
        for oh in range(ho):
            for ow in range(wo):
                hh, ww = s * oh + y0 - p, s * ow + x0 - p
                inside = 0 <= hh < hi and 0 <= ww < wi
                want = I[hh, ww, k % ci, :].astype(np.float64) if inside else np.zeros(b)
                assert np.array_equal(O[k, oh, ow, :], want)


@pytest.mark.parametrize("case", CASES)
def test_all_ones_count_taps(case):
    kn, kh, kw, ci, hi, wi, b, s, p = case
    F = np.ones((kn, kh, kw, ci), dtype=np.float32, order="F")
    I = np.ones((hi, wi, ci, b), dtype=np.float32, order="F")
    O = oc.conv_direct(F, I, s, p)
    ho, wo = O.shape[1], O.shape[2]
    for oh in range(ho):
        ny = sum(1 for y in range(kh) if 0 <= s * oh + y - p < hi)
        for ow in range(wo):
            nx = sum(1 for x in range(kw) if 0 <= s * ow + x - p < wi)
            assert (O[:, oh, ow, :] == ci * ny * nx).all()


def test_points_equal_direct_bitwise():
    case = CASES[1]
    kn, kh, kw, ci, hi, wi, b, s, p = case
    F, I = tensors(case, 17)
    O = oc.conv_direct(F, I, s, p)
    rng = synth.rng_for(18)
    pts = np.stack([rng.integers(0, d, 200) for d in O.shape], axis=1)
    got = oc.conv_points(F, I, pts, s, p)
    assert np.array_equal(got, O[tuple(pts.T)])


def test_thread_count_does_not_change_bits():
    case = (4, 3, 3, 3, 12, 10, 5, 2, 1)
    F, I = tensors(case, 19)
    old = oc.get_threads()
    try:
        oc.set_threads(1)
        a = oc.conv_direct(F, I, 2, 1)
        oc.set_threads(4)
        c = oc.conv_direct(F, I, 2, 1)
    finally:
        oc.set_threads(old)
    assert np.array_equal(a, c)


def test_rejects_mismatched_channels():
    F = sc.filter_tensor(2, 3, 3, 2, 1)
    I = sc.input_tensor(5, 5, 3, 1, 1)
    with pytest.raises(ValueError):
        oc.conv_direct(F, I)
