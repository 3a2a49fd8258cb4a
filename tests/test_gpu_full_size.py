"""Full-size parity at the benchmarked configurations: n = 16384 Gaussian fp64
(panel widths 128 and 256), n = 8192 graded fp64 and fp32, against the
oracle's complete results stored in ``tests/golden/full_*.npz`` (written by
``tests/golden/make_full_size.py``, which calls only the oracle; the oracle
takes minutes at these sizes).

Per workload, following the parity rules:
* the regenerated input is checked against the stored sample of the one the
  oracle factored;
* ipiv: bit-exact over all n entries, or, at the first split, the GPU's pivot
  is the oracle's runner-up within the near-tie margin (1 - 64 n eps); only
  earlier steps are then compared, rows taken in their order before the split;
* every alpha, and whole stored columns of L: normwise within 1e-10 (fp64);
  fp32: per column within max(1e-4, twice the fp32 oracle's own distance from
  the fp64 oracle in that column), alpha within max(1e-4, twice that distance);
* every multiplier through two fixed projections M z and M^T z (M = all
  multipliers), within what the normwise bar allows (tol * ||z||_1);
* log|Pf| within 1e-9 relative and the same sign (fp32: against the fp64
  oracle at 1e-4), and 2 log|Pf| against the device's slogdet(X) (det = Pf^2);
* |L| <= 1, finite factors, and the randomized residual estimate <= 10.
The even-step Pfaffian at n = 16384 is compared with the stored Pfaffian too.
"""
from __future__ import annotations

import os
import sys

import numpy as np
import pytest
import torch

from gpu_util import device_colmajor, host_packed, residual_probe

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))
from make_full_size import PROJ_SEED, WORKLOADS, make_input, undo_exchanges  # noqa: E402

import synth  # noqa: E402

pytestmark = pytest.mark.gpu


def lt():
    import paper_2005_06410_amd as m
    return m


def golden(name):
    path = os.path.join(HERE, "golden", f"full_{name}.npz")
    with np.load(path, allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


def regenerate(name, g):
    X = make_input(WORKLOADS[name])
    stride = int(g["sample_stride"])
    sample = np.ascontiguousarray(X.ravel()[::stride])
    assert np.array_equal(sample.view(np.uint8), np.ascontiguousarray(g["input_sample"]).view(np.uint8)), \
        "regenerated input differs from the one the oracle factored"
    return X


def split_point(ipiv, g, n, eps):
    """Columns that can be compared: all (n - 1) when the pivots agree, else
    the steps before the first split, which must be a near-tie."""
    d = np.nonzero(ipiv != g["ipiv"])[0]
    if not len(d):
        return n - 1, n
    kstar = int(d[0])
    k = kstar - 1                                   # ipiv[k+1] is step k's pivot
    assert int(ipiv[kstar]) == int(g["runner"][k]) and \
        g["runner_mag"][k] >= (1 - 64 * n * eps) * g["best"][k], \
        f"pivot split at step {k} is not a near-tie: gpu {ipiv[kstar]}, oracle {g['ipiv'][kstar]}"
    return k, kstar


def check_workload(name, nb):
    spec = WORKLOADS[name]
    n, dtype = spec["n"], spec["dtype"]
    fp32 = dtype == np.float32
    eps = np.finfo(dtype).eps
    g = golden(name)
    print(f"[full] {name} nb={nb}: input", flush=True)
    X = regenerate(name, g)
    flat, A = device_colmajor(X)
    print(f"[full] {name} nb={nb}: factor", flush=True)
    ip = lt().factor(A, nb=nb)
    logabs, sign = lt().pfaffian(A, ip)
    torch.cuda.synchronize()
    lt().device_status()
    ipiv = ip.cpu().numpy()
    logabs, sign = float(logabs.item()), int(sign.item())
    ncols, kstar = split_point(ipiv, g, n, eps)
    print(f"[full] {name} nb={nb}: pivots agree on {kstar} of {n}", flush=True)

    # alpha
    a_gpu = torch.diagonal(A, -1).double().cpu().numpy()
    a_ref = g["alpha"].astype(np.float64)
    tol_a = max(1e-4, 2.0 * float(g["drift_a"])) if fp32 else 1e-10
    if ncols > 0:
        ea = np.abs(a_gpu[:ncols] - a_ref[:ncols]).max() / np.abs(a_ref[:ncols]).max()
        assert ea <= tol_a, f"alpha normwise error {ea:.3e} > {tol_a:.1e}"
    if kstar == n:
        assert abs(a_gpu[n - 2] - a_ref[n - 2]) <= tol_a * np.abs(a_ref).max()

    # whole stored columns of L, rows in their order before any split
    off = 0
    worst = 0.0
    for c in g["col_index"]:
        c = int(c)
        ref = np.zeros(n)
        ref[c + 1:] = g["cols"][off:off + n - c - 1]
        off += n - c - 1
        if c >= ncols:
            continue
        got = np.zeros(n)
        got[c + 1:] = A[c + 1:, c].double().cpu().numpy()
        if kstar < n:
            ref = undo_exchanges(ref[:, None], g["ipiv"], ncols)[:, 0]
            got = undo_exchanges(got[:, None], ipiv, ncols)[:, 0]
        el = np.abs(got[c + 2:] - ref[c + 2:]).max() if c + 2 < n else 0.0
        tol = max(1e-4, 2.0 * float(np.nan_to_num(g["drift_col"][c], nan=np.nanmax(g["drift_col"])))) \
            if fp32 else 1e-10
        assert el <= tol, f"column {c}: L error {el:.3e} > {tol:.1e}"
        worst = max(worst, el)
    print(f"[full] {name} nb={nb}: alpha and columns ok (worst column error {worst:.2e})", flush=True)

    # every multiplier through M z and M^T z (pivots must agree for the rows to line up)
    M = torch.tril(A, -2).double()
    assert bool(torch.isfinite(M).all()) and float(M.abs().max()) <= 1.0
    if kstar == n:
        z = torch.from_numpy(synth.rng_for(int(g["proj_seed"])).standard_normal(n)).cuda()
        assert int(g["proj_seed"]) == PROJ_SEED
        lz = (M @ z).cpu().numpy()
        ltz = (M.t() @ z).cpu().numpy()
        z1 = float(z.abs().sum())
        tol = (max(1e-4, 2.0 * float(np.nanmax(g["drift_col"]))) if fp32 else 1e-10) * z1
        assert np.abs(lz - g["lz"]).max() <= tol and np.abs(ltz - g["ltz"]).max() <= tol
    del M

    # Pfaffian: against the oracle, and against det(X) = Pf(X)^2 on the device
    if fp32:
        assert sign == int(g["sign64"])
        assert abs(logabs - float(g["logabs64"])) <= 1e-4 * abs(float(g["logabs64"]))
    else:
        assert sign == int(g["sign"])
        assert abs(logabs - float(g["logabs"])) <= 1e-9 * abs(float(g["logabs"])), (logabs, float(g["logabs"]))
    Xd = torch.from_numpy(X.astype(np.float64)).cuda()
    sd, logdet = torch.linalg.slogdet(Xd)
    del Xd
    logdet = float(logdet.item())
    assert float(sd.item()) > 0
    assert abs(2 * logabs - logdet) <= (1e-4 if fp32 else 1e-9) * abs(logdet), (2 * logabs, logdet)

    # residual estimate
    packed = host_packed(flat, n, n)
    assert residual_probe(X, packed, ipiv) <= 10
    return logabs, sign


@pytest.mark.parametrize("nb", [128, 256])
def test_full_n16384_gauss_f64(nb):
    check_workload("n16384_gauss5_f64", nb)


def test_full_n8192_graded_f64():
    check_workload("n8192_graded4_f64", 128)


def test_full_n8192_graded_f32():
    check_workload("n8192_graded4_f32", 128)


def test_full_n16384_pfaffian_direct():
    name = "n16384_gauss5_f64"
    g = golden(name)
    X = regenerate(name, g)
    print("[full] even-step Pfaffian n=16384", flush=True)
    flat, A = device_colmajor(X)
    ip, logabs, sign = lt().pfaffian_direct(A, nb=128)
    torch.cuda.synchronize()
    lt().device_status()
    logabs, sign = float(logabs.item()), int(sign.item())
    # the Pfaffian is unique: the full reduction's value is the reference
    assert sign == int(g["sign"])
    assert abs(logabs - float(g["logabs"])) <= 1e-9 * abs(float(g["logabs"]))
