"""Write the oracle's results for the full-size factorization workloads.

The GPU parity tests at n = 16384 (Gaussian, fp64) and n = 8192 (graded,
fp64 and fp32) compare the library with these stored values, because the
oracle itself takes minutes at those sizes.  Everything here comes from
``oracle`` (the plain CPU reduction, run with OpenMP over the columns of its
rank-2 update, which gives the same bits as one thread) on inputs from
``synth``; numpy only lays the results out and forms fixed projections.

Stored per workload (``full_<name>.npz``):

* ``input_sample``: every 1000003rd entry of X (row-major), so a test can
  check that it regenerated the same input;
* ``ipiv`` (all n pivots), ``alpha`` (all n-1 subdiagonal entries of T);
* ``best``, ``runner``, ``runner_mag``: per column step, the pivot's
  magnitude and the runner-up row and magnitude (for the near-tie rule when
  a pivot sequence splits);
* ``cols`` / ``col_index``: whole packed columns c (rows c+1 .. n-1, i.e.
  alpha_c and the multipliers L(c+2:, c+1)), concatenated;
* ``lz`` = M z and ``ltz`` = M^T z, M = the strict part below the first
  subdiagonal of the packed output (all multipliers), z ~ N(0,1) from
  ``synth.rng_for(PROJ_SEED)``: every multiplier enters these sums;
* ``logabs``, ``sign``: the Pfaffian from the factors;
* fp32 only: ``logabs64``/``sign64`` from the fp64 oracle on the same
  (fp32-rounded) input; ``agree_steps``, the column steps before the fp32 and
  fp64 oracles' pivots first differ; over those columns ``drift_a``, the
  normwise distance of the fp32 oracle's alphas from the fp64 oracle's, and
  ``drift_col[c]``, the largest distance of its multipliers in column c, both
  sides' rows taken in their order before that first split (NaN from
  ``agree_steps`` on): how far fp32 arithmetic itself moves each column of
  these factors.

Usage: ``python tests/golden/make_full_size.py [name ...]`` (all by default).
It checks 2 log|Pf| against numpy's slogdet before writing.
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

PROJ_SEED = 777
SAMPLE_STRIDE = 1000003

WORKLOADS = {
    "n16384_gauss5_f64": dict(n=16384, kind="gauss", seed=5, dtype=np.float64,
                              cols=[0, 127, 128, 4095, 8191, 12287, 16000]),
    "n8192_graded4_f64": dict(n=8192, kind="graded", seed=4, dtype=np.float64,
                              cols=[0, 127, 128, 2047, 4095, 6143, 8000]),
    "n8192_graded4_f32": dict(n=8192, kind="graded", seed=4, dtype=np.float32,
                              cols=[0, 127, 128, 2047, 4095, 6143, 8000]),
}


def make_input(spec) -> np.ndarray:
    n, seed = spec["n"], spec["seed"]
    if spec["kind"] == "gauss":
        X = synth.skew_gauss(n, seed)
    elif spec["kind"] == "graded":
        X = synth.skew_graded(n, seed)
    else:
        raise ValueError(spec["kind"])
    return X.astype(spec["dtype"])


def undo_exchanges(cols: np.ndarray, ipiv: np.ndarray, k0: int) -> np.ndarray:
    """Rows of the multiplier columns ``cols`` (n x c, c <= k0) as they stood
    before column step k0: the exchanges (s+1, ipiv[s+1]) of the steps
    s >= k0 carried those rows along, and are undone here in reverse order."""
    out = cols.copy()
    n = out.shape[0]
    for s in range(n - 3, k0 - 1, -1):
        a, b = s + 1, int(ipiv[s + 1])
        if a != b:
            out[[a, b]] = out[[b, a]]
    return out


def projections(packed: np.ndarray, n: int):
    z = synth.rng_for(PROJ_SEED).standard_normal(n)
    M = np.tril(packed.astype(np.float64), -2)
    return M @ z, M.T @ z


def write(name: str) -> str:
    spec = WORKLOADS[name]
    n = spec["n"]
    t0 = time.time()
    X = make_input(spec)
    print(f"[{name}] input ready ({time.time() - t0:.1f} s)", flush=True)
    packed, ipiv, best, runner, rmag = oracle.ltlt_trace(X)
    print(f"[{name}] oracle done ({time.time() - t0:.1f} s, {oracle.get_threads()} threads)", flush=True)
    logabs, sign = oracle.pfaffian_packed(packed, ipiv)
    alpha = np.diagonal(packed, -1).copy()
    cols = [packed[c + 1:, c] for c in spec["cols"]]
    lz, ltz = projections(packed, n)
    out = dict(input_sample=X.ravel()[::SAMPLE_STRIDE].copy(), ipiv=ipiv, alpha=alpha, best=best,
               runner=runner, runner_mag=rmag, col_index=np.array(spec["cols"], dtype=np.int64),
               cols=np.concatenate(cols), lz=lz, ltz=ltz, logabs=np.float64(logabs), sign=np.int32(sign),
               proj_seed=np.int64(PROJ_SEED), sample_stride=np.int64(SAMPLE_STRIDE))
    Xd = X.astype(np.float64)
    if spec["dtype"] == np.float32:
        p64, i64 = oracle.ltlt(Xd)
        l64, s64 = oracle.pfaffian_packed(p64, i64)
        d = np.nonzero(i64 != ipiv)[0]
        agree = int(d[0]) - 1 if len(d) else n - 2         # steps before the first split
        nc = max(agree, 0)
        u32 = undo_exchanges(packed[:, :nc].astype(np.float64), ipiv, nc)
        u64 = undo_exchanges(p64[:, :nc], i64, nc)
        diff = np.abs(np.tril(u32 - u64, -2))
        drift_col = np.full(n - 1, np.nan)
        drift_col[:nc] = diff.max(axis=0) if nc else drift_col[:0]
        a32, a64 = alpha[:nc].astype(np.float64), np.diagonal(p64, -1)[:nc]
        d_a = float(np.abs(a32 - a64).max() / np.abs(a64).max()) if nc else 0.0
        out.update(logabs64=np.float64(l64), sign64=np.int32(s64), drift_col=drift_col,
                   drift_a=np.float64(d_a), agree_steps=np.int64(agree))
        q = np.quantile(drift_col[:nc], [0.5, 0.9, 0.99]) if nc else [0, 0, 0]
        print(f"[{name}] fp64 reference: pivots agree for {agree} steps; alpha drift {d_a:.3e}; "
              f"column drift median {q[0]:.2e} p90 {q[1]:.2e} p99 {q[2]:.2e} max {np.nanmax(drift_col):.2e}",
              flush=True)
        ref_logabs = l64
    else:
        ref_logabs = logabs
    s_det, logdet = np.linalg.slogdet(Xd)
    rel = abs(2.0 * ref_logabs - logdet) / abs(logdet)
    print(f"[{name}] log|Pf| {ref_logabs:.12f}  slogdet/2 {logdet / 2:.12f}  rel {rel:.2e}", flush=True)
    tol = 1e-9
    assert s_det > 0 and rel <= tol, "oracle Pfaffian disagrees with det = Pf^2"
    path = os.path.join(HERE, f"full_{name}.npz")
    np.savez(path, **out)
    print(f"[{name}] wrote {path} ({os.path.getsize(path) / 1e6:.2f} MB, {time.time() - t0:.1f} s)", flush=True)
    return path


def main(argv):
    names = argv or list(WORKLOADS)
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    oracle.set_threads(threads)
    for name in names:
        write(name)


if __name__ == "__main__":
    main(sys.argv[1:])
