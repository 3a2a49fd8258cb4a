"""GPU parity of the blocked factorization, the Pfaffian and the trailing
update against the CPU oracle (same seeded inputs, same precision).

Inputs follow the workloads: Gaussian skew matrices (strict upper iid N(0,1)),
graded ones (N(0,1) * 10^U(-3,3)), 4x4-block-diagonal ones, at sizes that
span several panels and tiles with ragged tails, plus the full sizes
n = 8192 and 16384 checked on sampled outputs (the first column steps against
the oracle run for those steps only) and on size-independent properties."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import compare_factors, device_colmajor, gpu_factor, host_packed
from truths import pf_closed4

pytestmark = pytest.mark.gpu


def lt():
    import paper_2005_06410_amd as m
    return m


def check_pf(X, packed, ipiv, logabs, sign, dtype, ref_pf=None):
    if ref_pf is None:
        ref_pf = oracle.pfaffian_packed(packed.astype(dtype), ipiv)  # same factors, oracle arithmetic
    rl, rs = ref_pf
    assert sign == rs
    if rs != 0:
        assert abs(logabs - rl) <= 1e-9 * max(abs(rl), 1.0), (logabs, rl)


# --------------------------------------------------------------------------
@pytest.mark.parametrize("n,nb", [(3, 1), (4, 1), (5, 2), (8, 3), (17, 4), (33, 8), (64, 16), (100, 32),
                                  (129, 128), (200, 64), (255, 7), (300, 128), (513, 64)])
def test_parity_gauss_fp64(n, nb):
    X = synth.skew_gauss(n, 100 + n)
    packed, ipiv, logabs, sign, _ = gpu_factor(X, nb=nb)
    info = compare_factors(X, packed, ipiv, np.float64)
    assert info["first_pivot_mismatch"] == n
    assert oracle.residual(X, packed, ipiv) <= 10
    ref = oracle.pfaffian(X)
    check_pf(X, packed, ipiv, logabs, sign, np.float64, ref)


@pytest.mark.parametrize("n,nb", [(64, 8), (200, 32), (400, 128)])
def test_parity_graded_fp64(n, nb):
    X = synth.skew_graded(n, 7 + n)
    packed, ipiv, logabs, sign, _ = gpu_factor(X, nb=nb)
    compare_factors(X, packed, ipiv, np.float64)
    assert oracle.residual(X, packed, ipiv) <= 10
    check_pf(X, packed, ipiv, logabs, sign, np.float64, oracle.pfaffian(X))


@pytest.mark.parametrize("n,nb", [(50, 16), (257, 128), (600, 128)])
def test_parity_fp32(n, nb):
    X = synth.skew_gauss(n, 55 + n).astype(np.float32)
    packed, ipiv, logabs, sign, _ = gpu_factor(X, nb=nb)
    compare_factors(X, packed, ipiv, np.float32)
    assert oracle.residual(X, packed, ipiv) <= 10
    # fp32 factors: log|Pf| against the fp64 oracle on the same (rounded) input
    rl, rs = oracle.pfaffian(X.astype(np.float64))
    assert sign == rs
    if rs != 0:
        assert abs(logabs - rl) <= 1e-4 * abs(rl)
    else:
        assert logabs == -math.inf


def test_config_n256_b32():
    X = synth.skew_gauss(256, 1)
    packed, ipiv, logabs, sign, _ = gpu_factor(X, nb=32)
    compare_factors(X, packed, ipiv, np.float64)
    assert oracle.residual(X, packed, ipiv) <= 10
    check_pf(X, packed, ipiv, logabs, sign, np.float64, oracle.pfaffian(X))


def test_config_n2048_b64():
    X = synth.skew_gauss(2048, 2)
    packed, ipiv, logabs, sign, _ = gpu_factor(X, nb=64)
    compare_factors(X, packed, ipiv, np.float64)
    assert oracle.residual(X, packed, ipiv) <= 10
    s, logdet = np.linalg.slogdet(X)
    assert abs(2 * logabs - logdet) <= 1e-9 * abs(logdet)
    check_pf(X, packed, ipiv, logabs, sign, np.float64, oracle.pfaffian(X))


def test_config_n2048_blockdiag4():
    n = 2048
    X = synth.skew_blockdiag4(n, 3)
    packed, ipiv, logabs, sign, _ = gpu_factor(X, nb=64)
    compare_factors(X, packed, ipiv, np.float64)
    ref_log, ref_sign = 0.0, 1
    for b in range(n // 4):
        pf = pf_closed4(X[4 * b:4 * b + 4, 4 * b:4 * b + 4])
        ref_log += math.log(abs(pf))
        ref_sign *= int(np.sign(pf))
    assert sign == ref_sign
    assert abs(logabs - ref_log) <= 1e-9 * abs(ref_log)
    # zero columns: alpha exactly 0, no exchange, multipliers exactly 0
    for b in range(n // 4 - 1):
        k = 4 * b + 3
        assert packed[k + 1, k] == 0.0 and ipiv[k + 1] == k + 1
        assert np.all(packed[k + 2:, k] == 0.0)


# --------------------------------------------------------------------------
@pytest.mark.parametrize("n", [0, 1, 2, 3])
def test_tiny_orders(n):
    X = synth.skew_gauss(n, 9) if n else np.zeros((0, 0))
    packed, ipiv, logabs, sign, _ = gpu_factor(X)
    ref_p, ref_i = oracle.ltlt(X)
    assert np.array_equal(ipiv, ref_i)
    assert np.allclose(packed, ref_p, rtol=1e-14, atol=0)
    if n == 2:
        assert packed[1, 0] == X[1, 0]
    ref = oracle.pfaffian(X)
    assert sign == ref[1]
    if ref[1]:
        assert logabs == pytest.approx(ref[0], rel=1e-14, abs=1e-14)
    else:
        assert logabs == -math.inf


def test_lda_larger_than_n_and_padding_untouched():
    n, lda = 150, 163
    X = synth.skew_gauss(n, 17)
    packed, ipiv, logabs, sign, flat = gpu_factor(X, nb=32, lda=lda, fill=np.nan)
    buf = flat.cpu().numpy().reshape(n, lda)
    assert np.all(np.isnan(buf[:, n:]))                # rows n..lda-1 never touched
    compare_factors(X, packed, ipiv, np.float64)


@pytest.mark.parametrize("n,nb", [(130, 32), (700, 128)])
def test_diagonal_and_upper_never_read_or_written(n, nb):
    X = synth.skew_gauss(n, 18)
    flat, A = device_colmajor(X)
    A.diagonal().fill_(float("nan"))
    up = torch.triu(torch.ones(n, n, dtype=torch.bool, device="cuda"), 1)
    A.masked_fill_(up, float("inf"))                   # sentinels: must not be read
    ipiv = lt().factor(A, nb=nb)
    torch.cuda.synchronize()
    assert torch.isnan(A.diagonal()).all()
    assert torch.isinf(A[up]).all()                     # and not written
    packed = host_packed(flat, n, n)
    compare_factors(X, packed, ipiv.cpu().numpy(), np.float64)


def test_row_major_tensor_is_rejected():
    X = torch.zeros(8, 8, dtype=torch.float64, device="cuda")
    with pytest.raises(ValueError):
        lt().factor(X.t().contiguous())  # stride(0) = 8: row-major
    with pytest.raises(ValueError):
        lt().factor(X[:, :7].t())


def test_zero_matrix_and_tridiagonal_input():
    n = 70
    packed, ipiv, logabs, sign, _ = gpu_factor(np.zeros((n, n)), nb=16)
    assert np.all(packed == 0) and list(ipiv) == list(range(n)) and sign == 0
    rng = synth.rng_for(19)
    X = np.zeros((n, n))
    X[np.arange(1, n), np.arange(n - 1)] = rng.standard_normal(n - 1)
    X = X - X.T
    packed, ipiv, logabs, sign, _ = gpu_factor(X, nb=16)
    assert list(ipiv) == list(range(n))
    assert np.array_equal(packed, np.tril(X, -1))


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_exact_invariants_scaling_and_negation(dtype):
    n = 300
    X = synth.skew_gauss(n, 23).astype(dtype)
    p0, i0, l0, s0, _ = gpu_factor(X, nb=64)
    p1, i1, l1, s1, _ = gpu_factor(X * dtype(8.0), nb=64)
    p2, i2, l2, s2, _ = gpu_factor(-X, nb=64)
    sub = np.arange(1, n), np.arange(n - 1)
    low = np.tril(np.ones((n, n), bool), -2)
    assert np.array_equal(i0, i1) and np.array_equal(i0, i2)
    assert np.array_equal(p1[sub], p0[sub] * dtype(8.0))
    assert np.array_equal(p2[sub], -p0[sub])
    assert np.array_equal(p1[low], p0[low]) and np.array_equal(p2[low], p0[low])


def test_bitwise_deterministic():
    X = synth.skew_graded(700, 29)
    a = gpu_factor(X, nb=128)
    b = gpu_factor(X, nb=128)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[2] == b[2]


@pytest.mark.parametrize("nb", [1, 17, 64, 200, 256])
def test_panel_widths(nb):
    X = synth.skew_gauss(520, 31)
    packed, ipiv, logabs, sign, _ = gpu_factor(X, nb=nb)
    compare_factors(X, packed, ipiv, np.float64)


# --------------------------------------------------------------------------
@pytest.mark.parametrize("m,K,off,dtype", [(2, 1, 0, np.float64), (100, 5, 0, np.float64),
                                           (129, 129, 7, np.float64), (300, 33, 20, np.float64),
                                           # fp64 halves of 128 x 128 tiles: one, two, three
                                           # and more operand chunks (K = 8, 9, 16, 17, 25),
                                           # an empty second half (m = 64, 130), every wave
                                           # of a diagonal half above the diagonal (m = 193)
                                           (64, 8, 3, np.float64), (130, 9, 5, np.float64),
                                           (193, 16, 9, np.float64), (256, 17, 0, np.float64),
                                           (385, 25, 12, np.float64), (700, 257, 33, np.float64),
                                           (257, 17, 11, np.float32), (128, 4, 3, np.float32)])
def test_skew_update_parity(m, K, off, dtype):
    rng = synth.rng_for(m * 1000 + K)
    N = m + off
    S = synth.skew_gauss(N, m + K).astype(dtype)
    Lx = rng.standard_normal((m, K)).astype(dtype)
    Bt = rng.standard_normal((m, K)).astype(dtype)
    # perm: identity on the block except a few rows that read from the `off`
    # rows/columns before the block (as the panel's displaced indices do)
    perm = np.arange(m, dtype=np.int32)
    if off:
        pos = rng.choice(m, size=min(off, m), replace=False)
        perm[pos] = rng.choice(np.arange(-off, 0), size=len(pos), replace=False).astype(np.int32)
    flat, Cv = device_colmajor(S)
    Ld = torch.from_numpy(np.asfortranarray(Lx)).cuda()
    Bd = torch.from_numpy(np.asfortranarray(Bt)).cuda()
    Ld = Ld.t().contiguous().t()
    Bd = Bd.t().contiguous().t()
    pd = torch.from_numpy(perm).cuda()
    lt().skew_update(Cv, Ld, Bd, perm=pd, offset=off)
    torch.cuda.synchronize()
    got = flat.cpu().numpy().reshape(N, N).T            # (i, j) indexing
    Sfull = S.astype(np.float64)
    ref_blk = oracle.skew_update(Sfull, np.pad(Lx.astype(np.float64), ((off, 0), (0, 0))),
                                 np.pad(Bt.astype(np.float64), ((off, 0), (0, 0))),
                                 np.concatenate([np.arange(off), perm + off]).astype(np.int64))
    g = got[off:, off:].astype(np.float64)
    r = ref_blk[off:, off:]
    iu = np.triu_indices(m, 0)
    il = np.tril_indices(m, -1)
    tol = 1e-12 if dtype == np.float64 else 2e-5
    scale = np.abs(r).max()
    assert np.abs(g[il] - r[il]).max() <= tol * scale * max(1, K) ** 0.5
    assert np.array_equal(got[off:, off:][iu], S[off:, off:][iu])   # diagonal and upper untouched
    # outside the block nothing changed
    assert np.array_equal(got[:off, :], S[:off, :]) and np.array_equal(got[:, :off], S[:, :off])


@pytest.mark.parametrize("layout", ["aligned", "offset1", "odd_ld"])
def test_skew_update_operand_layouts(layout):
    """fp64 operands whose columns start 16-byte aligned are copied straight
    into LDS; an odd start or an odd leading dimension takes the register
    path.  Both must give the oracle's result (m = 258: three tile rows and a
    ragged last one; K = 130: a ragged last K chunk)."""
    m, K = 258, 130
    rng = synth.rng_for(4242)
    S = synth.skew_gauss(m, 77)
    Lx = rng.standard_normal((m, K))
    Bt = rng.standard_normal((m, K))
    flat, Cv = device_colmajor(S)

    def place(X):
        if layout == "aligned":
            return torch.from_numpy(np.asfortranarray(X)).cuda().t().contiguous().t()
        ld = m + 1 if layout == "odd_ld" else m
        start = 1 if layout == "offset1" else 0
        buf = torch.zeros(start + ld * K + 1, dtype=torch.float64, device="cuda")
        v = buf[start:start + ld * K].view(K, ld)[:, :m]
        v.copy_(torch.from_numpy(np.ascontiguousarray(X.T)).cuda())
        return v.t()

    Ld, Bd = place(Lx), place(Bt)
    assert Ld.stride() == (1, m + 1 if layout == "odd_ld" else m)
    lt().skew_update(Cv, Ld, Bd)
    torch.cuda.synchronize()
    got = flat.cpu().numpy().reshape(m, m).T
    ref = oracle.skew_update(S, Lx, Bt, np.arange(m, dtype=np.int64))
    il = np.tril_indices(m, -1)
    iu = np.triu_indices(m, 0)
    assert np.abs(got[il] - ref[il]).max() <= 1e-12 * np.abs(ref).max() * K ** 0.5
    assert np.array_equal(got[iu], S[iu])


# --------------------------------------------------------------------------
@pytest.mark.parametrize("n,batch,dtype", [(64, 8192, np.float64), (64, 8192, np.float32), (64, 300, np.float32), (1, 5, np.float64),
                                           (2, 5, np.float64), (7, 33, np.float64), (40, 129, np.float64),
                                           # orders at the 16-step block boundaries of the batched kernel
                                           (16, 65, np.float64), (17, 65, np.float64), (18, 65, np.float64),
                                           (32, 65, np.float64), (33, 65, np.float64), (48, 65, np.float64),
                                           (49, 65, np.float64), (50, 65, np.float64), (63, 65, np.float64),
                                           (33, 65, np.float32)])
def test_batched_parity(n, batch, dtype):
    Xs = synth.skew_batch(n, batch, 6 << 32 if n == 64 else 99).astype(dtype)
    ref_p, ref_i, ref_l, ref_s = oracle.ltlt_batched(Xs)
    buf = np.ascontiguousarray(np.transpose(Xs, (0, 2, 1)))      # column-major per matrix
    d = torch.from_numpy(buf).cuda()
    A = d.as_strided((batch, n, n), (n * n, 1, n))
    ipiv, logabs, sign = lt().factor_batched(A)
    torch.cuda.synchronize()
    got = np.tril(np.transpose(d.cpu().numpy(), (0, 2, 1)), -1)
    gi = ipiv.cpu().numpy()
    mism = 0
    for b in range(batch):
        if not np.array_equal(gi[b], ref_i[b]):
            mism += 1
            compare_factors(Xs[b].astype(dtype), got[b], gi[b], dtype)
            continue
        tol = 1e-10 if dtype == np.float64 else 1e-4
        if n >= 2:
            scale = np.abs(ref_p[b]).max()
            assert np.abs(got[b].astype(np.float64) - ref_p[b]).max() <= tol * max(scale, 1e-300)
    assert mism <= max(1, batch // 1000)
    s = sign.cpu().numpy()
    la = logabs.cpu().numpy()
    assert np.array_equal(s, ref_s)
    ok = ref_s != 0
    if dtype == np.float64:
        assert np.all(np.abs(la[ok] - ref_l[ok]) <= 1e-9 * np.maximum(np.abs(ref_l[ok]), 1.0))
    else:
        # fp32 (the reading of the fp32 bar): against the fp64 oracle on the
        # same rounded input, within 1e-4 relative or twice the fp32 oracle's
        # own distance from it, whichever is larger (a member with one small
        # alpha_2j puts the fp32 oracle itself past 1e-4 in about one of
        # 8192 Gaussian matrices)
        _, _, l64, s64 = oracle.ltlt_batched(Xs.astype(np.float64))
        ok = ok & (s64 != 0)
        bar = np.maximum(1e-4 * np.maximum(np.abs(l64[ok]), 1.0), 2.0 * np.abs(ref_l[ok] - l64[ok]))
        assert np.all(np.abs(la[ok] - l64[ok]) <= bar)
    # upper triangle and diagonal untouched by the batched path
    full = np.transpose(d.cpu().numpy(), (0, 2, 1))
    iu = np.triu_indices(n, 0)
    assert np.array_equal(full[:, iu[0], iu[1]], Xs[:, iu[0], iu[1]])


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_batched_padded_layout(dtype):
    """lda > n and a matrix stride past lda*n: the factors land in each
    matrix's strict lower triangle at its leading dimension, and the padding
    rows, the gaps between matrices, the diagonal and the upper triangle keep
    their sentinel values."""
    n, batch, lda = 40, 37, 47
    stride = lda * n + 13
    Xs = synth.skew_batch(n, batch, 4242).astype(dtype)
    ref_p, ref_i, ref_l, ref_s = oracle.ltlt_batched(Xs)
    sentinel = dtype(-7.25)
    flat = np.full(stride * batch, sentinel, dtype=dtype)
    for b in range(batch):
        M = np.full((n, lda), sentinel, dtype=dtype)     # M[c, r] = A(r, c): column-major with lda
        M[:, :n] = Xs[b].T
        flat[b * stride:b * stride + lda * n] = M.ravel()
    d = torch.from_numpy(flat.copy()).cuda()
    A = d.as_strided((batch, n, n), (stride, 1, lda))
    ipiv, logabs, sign = lt().factor_batched(A)
    torch.cuda.synchronize()
    out = d.cpu().numpy()
    gi = ipiv.cpu().numpy()
    tol = 1e-10 if dtype == np.float64 else 1e-4
    for b in range(batch):
        blk = out[b * stride:(b + 1) * stride]
        M = blk[:lda * n].reshape(n, lda)               # M[c, r] = A(r, c)
        got = np.tril(M[:, :n].T, -1)
        if np.array_equal(gi[b], ref_i[b]):
            assert np.abs(got.astype(np.float64) - ref_p[b]).max() <= tol * max(np.abs(ref_p[b]).max(), 1e-300)
        else:
            compare_factors(Xs[b], got, gi[b], dtype)
        assert np.all(M[:, n:] == sentinel)             # padding rows n .. lda-1
        assert np.all(blk[lda * n:] == sentinel)        # gap before the next matrix
        iu = np.triu_indices(n, 0)
        assert np.array_equal(M[:, :n].T[iu], Xs[b][iu])
    assert np.array_equal(sign.cpu().numpy(), ref_s)


def test_batched_zero_structured_matrices():
    """Zero-structured members of a batch: 4x4 block-diagonal matrices (every
    column step ties on zeros outside one block, and every k = 3 mod 4 column
    is exactly zero) and the zero matrix, beside Gaussian ones.  ipiv matches
    the oracle bit for bit, factors to 1e-10, Pf = the product of the blocks'
    closed-form 4x4 Pfaffians, and each matrix gives the same result as when
    it is factored alone (batch of one)."""
    n = 64
    Xs = synth.skew_batch(n, 48, 777)
    for b in range(0, 48, 3):
        Xs[b] = synth.skew_blockdiag4(n, 500 + b)
    Xs[1] = 0.0
    ref_p, ref_i, ref_l, ref_s = oracle.ltlt_batched(Xs)
    buf = np.ascontiguousarray(np.transpose(Xs, (0, 2, 1)))
    d = torch.from_numpy(buf).cuda()
    A = d.as_strided((48, n, n), (n * n, 1, n))
    ipiv, logabs, sign = lt().factor_batched(A)
    torch.cuda.synchronize()
    got = np.tril(np.transpose(d.cpu().numpy(), (0, 2, 1)), -1)
    gi, la, sg = ipiv.cpu().numpy(), logabs.cpu().numpy(), sign.cpu().numpy()
    assert np.array_equal(gi, ref_i)
    for b in range(48):
        scale = max(np.abs(ref_p[b]).max(), 1e-300)
        assert np.abs(got[b] - ref_p[b]).max() <= 1e-10 * scale
    assert np.array_equal(sg, ref_s)
    for b in range(0, 48, 3):                       # closed forms of the block-diagonal members
        pf = 1.0
        for q in range(n // 4):
            blk = Xs[b][4 * q:4 * q + 4, 4 * q:4 * q + 4]
            pf *= blk[0, 1] * blk[2, 3] - blk[0, 2] * blk[1, 3] + blk[0, 3] * blk[1, 2]
        assert sg[b] == np.sign(pf)
        assert abs(la[b] - np.log(abs(pf))) <= 1e-12 * max(abs(np.log(abs(pf))), 1.0)
    assert sg[1] == 0 and la[1] == -np.inf and np.all(gi[1] == np.arange(n))
    for b in (0, 1, 3):                             # alone vs in the batch
        d1 = torch.from_numpy(np.ascontiguousarray(Xs[b].T)).cuda()
        A1 = d1.as_strided((1, n, n), (n * n, 1, n))
        i1, l1, s1 = lt().factor_batched(A1)
        torch.cuda.synchronize()
        assert np.array_equal(np.tril(d1.cpu().numpy().T, -1), got[b])
        assert np.array_equal(i1.cpu().numpy()[0], gi[b]) and s1.item() == sg[b]


def _triu_rows(M, k, ch=8192):
    """torch.triu(M, k) built on row chunks: on this PyTorch build torch.triu of
    a tensor past 2^32 elements returns wrong entries (a quarter of a sample at
    66000^2), while every chunk here stays below 2^31."""
    out = torch.empty_like(M)
    for r0 in range(0, M.shape[0], ch):
        out[r0:r0 + ch] = torch.triu(M[r0:r0 + ch], k + r0)
    return out


@pytest.mark.parametrize("n,dtype", [(70000, torch.float64), (33000, torch.complex128)])
def test_large_order_default_width_fallback(n, dtype):
    """Orders past what the default width's panel holds on one device (real:
    n - 1 > 256 workgroups x 256 rows at nb = 128; complex: 256 x 128 rows):
    ltlt_factor narrows the width and factors them.  The input is generated
    on the device (its strict lower triangle is a seeded Gaussian buffer);
    checked by the pivot invariants and a two-probe residual estimate in the
    factor's precision, computed on the device (the oracle would take hours)."""
    elt = 16 if dtype == torch.complex128 else 8
    free, _ = torch.cuda.mem_get_info()
    if free < 2.6 * n * n * elt + 8e9:
        pytest.skip("needs about %.0f GB of free device memory" % (2.6 * n * n * elt / 1e9))
    dev = torch.device("cuda")
    gen = torch.Generator(device=dev)
    gen.manual_seed(n)
    buf = torch.randn(n * n, dtype=dtype, device=dev, generator=gen)
    R = buf.view(n, n)                              # R[c, i] = A(i, c)
    U = _triu_rows(R, 1)                            # X = U^T - U
    A = buf.as_strided((n, n), (1, n))
    ipiv = lt().factor(A)
    torch.cuda.synchronize()
    piv = ipiv.cpu().numpy()
    assert piv[0] == 0 and piv[n - 1] == n - 1
    assert np.all(piv[1:-1] >= np.arange(1, n - 1)) and np.all(piv < n)
    perm = np.arange(n)
    for i, j in enumerate(piv.tolist()):
        perm[i], perm[j] = perm[j], perm[i]
    perm_t = torch.from_numpy(perm).to(dev)
    Z = torch.randn(n, 2, dtype=dtype, device=dev, generator=gen)
    PtZ = torch.empty_like(Z)
    PtZ[perm_t] = Z                                 # P^T Z
    left = ((PtZ.T @ U).T - U @ PtZ)[perm_t]        # P X P^T Z
    normX = 2 ** 0.5 * torch.linalg.norm(U).item()
    if dtype == torch.float64:
        # the solve on the same factors: backward error against X
        b = torch.randn(2, n, dtype=dtype, device=dev, generator=gen).t()   # n x 2, column-major
        x = b.clone().t().contiguous().t()
        lt().solve(A, ipiv, x)
        torch.cuda.synchronize()
        Xx = (x.T @ U).T - U @ x
        absU_rows = torch.cat([U[r0:r0 + 8192].abs().sum(1) for r0 in range(0, n, 8192)])
        absU_cols = sum(U[r0:r0 + 8192].abs().sum(0) for r0 in range(0, n, 8192))
        normXinf = (absU_rows + absU_cols).max().item()     # largest row sum of |U^T - U|
        eps = torch.finfo(torch.float64).eps
        for c in range(2):
            be = (Xx[:, c] - b[:, c]).abs().max().item() / (normXinf * x[:, c].abs().max().item() * n * eps)
            assert be <= 10.0, be
        del b, x, Xx
    del U
    Lp = _triu_rows(R, 2)                           # Lp[c, r] = A(r, c) = L(r, c + 1), r >= c + 2
    alpha = torch.diagonal(R, 1)                    # alpha_k = A(k + 1, k)
    V = Z.clone()
    V[1:] += (Lp @ Z)[:-1]                          # L^T Z
    TV = torch.zeros_like(V)
    TV[1:] += alpha[:, None] * V[:-1]               # T(k + 1, k) = alpha_k
    TV[:-1] -= alpha[:, None] * V[1:]               # T(k, k + 1) = -alpha_k
    sh = torch.zeros_like(TV)
    sh[:-1] = TV[1:]
    right = TV + (sh.T @ Lp).T                      # L (T L^T Z)
    eps = torch.finfo(torch.float64).eps
    est = torch.linalg.norm(left - right).item() / 2 ** 0.5 / (n * eps * normX)
    assert est <= 10.0, est
    assert torch.isfinite(alpha).all()


@pytest.mark.parametrize("kind", ["factor", "pfaffian_direct", "complex"])
def test_panel_launch_modes_agree(kind):
    """The panels' ordinary launch (default) and the cooperative launch give
    bit-identical results (only the launch path differs)."""
    lib = lt()
    n = 1030
    X = synth.skew_gauss_complex(n, 31) if kind == "complex" else synth.skew_gauss(n, 31)
    out = []
    try:
        for coop in (False, True):
            lib.set_cooperative_panels(coop)
            flat, A = device_colmajor(X)
            if kind == "pfaffian_direct":
                ipiv, la, sg = lib.pfaffian_direct(A, nb=64)
                res = [flat, ipiv, la, sg]
            else:
                ipiv = lib.factor(A)
                la, sg = lib.pfaffian(A, ipiv)
                res = [flat, ipiv, la, sg]
            torch.cuda.synchronize()
            lib.device_status()
            out.append([r.cpu().clone() for r in res])
    finally:
        lib.set_cooperative_panels(False)
    for a, b in zip(*out):
        assert torch.equal(a, b)


@pytest.mark.parametrize("n,reps", [(1000, 40), (16384, 3)])
def test_repeated_runs_bit_identical(n, reps):
    """Back-to-back factorizations with the default panel launch finish
    inside the panels' bounded waits and give bit-identical factors and
    pivots every time (the grid exchange fixes the reduction order)."""
    lib = lt()
    X = synth.skew_gauss(n, 11)
    src, _ = device_colmajor(X)
    w = torch.empty_like(src)
    A = w.as_strided((n, n), (1, n))
    ipiv = torch.empty(n, dtype=torch.int32, device="cuda")
    ref = None
    for _ in range(reps):
        w.copy_(src)
        lib.factor(A, ipiv=ipiv)
        torch.cuda.synchronize()
        lib.device_status()
        if ref is None:
            ref = (w.clone(), ipiv.clone())
        else:
            assert torch.equal(w, ref[0]) and torch.equal(ipiv, ref[1])


# --------------------------------------------------------------------------
@pytest.mark.parametrize("dtype,published", [("f64", 78.6), ("f32", 157.3)])
def test_mfma_probe_rate(dtype, published):
    """The measured register-only MFMA loop rate lies between half of the
    published dense peak and the peak itself (plus clock headroom)."""
    rate = lt().mfma_probe(dtype, iters=4000)
    assert 0.5 * published <= rate <= 1.1 * published, rate


def test_binding_rejects_mismatched_arguments():
    """Host tensors, other dtypes and short pivot vectors are refused by the
    binding before any kernel sees their pointers."""
    n = 16
    flat, A = device_colmajor(synth.skew_gauss(n, 3))
    with pytest.raises(ValueError):
        lt().factor(A, ipiv=torch.empty(n, dtype=torch.int32))            # host tensor
    with pytest.raises(ValueError):
        lt().factor(A, ipiv=torch.empty(n, dtype=torch.int64, device="cuda"))
    with pytest.raises(ValueError):
        lt().factor(A, ipiv=torch.empty(n - 1, dtype=torch.int32, device="cuda"))
    ipiv = lt().factor(A)
    with pytest.raises(ValueError):
        lt().pfaffian(A, ipiv.cpu())
    with pytest.raises(ValueError):
        lt().solve(A, ipiv, torch.ones(n, dtype=torch.float32, device="cuda"))
    with pytest.raises(ValueError):
        lt().solve(A, ipiv.cpu(), torch.ones(n, dtype=torch.float64, device="cuda"))
    C = torch.zeros((8, 8), dtype=torch.float64, device="cuda").t().contiguous().t()
    Lx = torch.zeros((8, 3), dtype=torch.float32, device="cuda").t().contiguous().t()
    with pytest.raises(ValueError):
        lt().skew_update(C, Lx, Lx)                                    # operands of another dtype
    Lx64 = torch.zeros((8, 3), dtype=torch.float64, device="cuda").t().contiguous().t()
    with pytest.raises(ValueError):
        lt().skew_update(C, Lx64, Lx64, offset=1)                      # block past the end of C
    torch.cuda.synchronize()
