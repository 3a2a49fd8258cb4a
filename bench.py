"""Benchmark: LTL^T factorization GFLOP/s (n^3/3) of one n=16384 fp64
skew-symmetric matrix on one MI355X, plus the roofline of the dominant kernel
(the trailing update) and the CPU oracle timed on a bounded sample.

One step = one whole factorization (panel, trailing update, commit and the
final row ordering of every block) plus the Pfaffian, on a matrix already
resident in HBM.  Before each step the matrix is restored from a pristine
device copy (outside the timed events: the factorization works in place).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--nb 128]
                       [--n 16384] [--dtype f64|f32] [--no-cpu-baseline]
                       [--workload factor|batched|pfaffian|solve|complex|cpu-oracle] [--nrhs R]
Prints one JSON line.  `--workload batched` instead times the batched path
(8192 independent n=64 matrices, factors + Pfaffians) against HBM bandwidth;
`--workload pfaffian` the Pfaffian by the even column steps alone;
`--workload solve` the solve X x = b with the factors (R right-hand sides)
against HBM bandwidth; `--workload complex` the factorization + Pfaffian of a
complex128 (or, with --dtype f32, complex64) skew-symmetric matrix;
`--workload cpu-oracle` runs the whole CPU oracle at --n on the host's cores
(no GPU) and prints its rate; `--workload convgemm` times the paper's own
operator, CONVGEMM (convolution as one GEMM with im2col folded into operand
staging), over the five AlexNet convolution layers of the paper's Table 2 at
batch --conv-batch (default 80), in fp32 TFLOP/s.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP64_PEAK_TF = 78.6      # MI355X dense FP64 matrix peak (AMD spec)
FP32_PEAK_TF = 157.3     # MI355X dense FP32 matrix peak
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--n", type=int, default=16384)
    ap.add_argument("--nb", type=int, default=None, help="panel width (default 128)")
    ap.add_argument("--dtype", choices=["f64", "f32"], default="f64")
    ap.add_argument("--seed", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--workload", choices=["factor", "batched", "pfaffian", "solve", "complex", "cpu-oracle",
                                           "convgemm"],
                    default="factor")
    ap.add_argument("--conv-batch", type=int, default=80, help="convgemm workload: batch size b")
    ap.add_argument("--tile", default="0,0", help="convgemm workload: workgroup tile mt,nt (0,0 = automatic)")
    ap.add_argument("--conv-path", type=int, default=0,
                    help="convgemm workload: 0 automatic, 1 LDS-staged gather, 2 register-direct")
    ap.add_argument("--nrhs", type=int, default=1)
    ap.add_argument("--batch", type=int, default=8192)
    ap.add_argument("--input", choices=["gauss", "graded", "blockdiag4"], default="gauss",
                    help="factor workload input: strict upper iid N(0,1); times 10^U(-3,3) per entry; "
                         "or 4x4 Gaussian skew blocks on the diagonal")
    return ap.parse_args()


def host_info():
    """The host the CPU baseline ran on: logical CPUs, the CPUs this process
    may use, the CPU model and OMP_NUM_THREADS."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "cpus_allowed": len(os.sched_getaffinity(0)), "cpu_model": model,
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


def oracle_threads():
    """Threads for the oracle's OpenMP loop: OMP_NUM_THREADS when set (the
    share of the host this process is given), else every CPU it may use."""
    v = os.environ.get("OMP_NUM_THREADS", "")
    return int(v) if v.isdigit() and int(v) > 0 else len(os.sched_getaffinity(0))


def _oracle_prefix_rate(buf, n, target_s, threads):
    """Run the oracle's first column steps on a copy of ``buf`` with
    ``threads`` threads, about ``target_s`` seconds; returns (steps, seconds,
    nominal flops) with step k counting (n-k-2)^2 (the n^3/3 convention)."""
    import oracle
    oracle.set_threads(threads)
    b = buf.copy()
    t0 = time.perf_counter()
    oracle.ltlt_colmajor(b, n, 4)                     # calibration: four steps
    t4 = (time.perf_counter() - t0) / 4
    steps = int(max(1, min(n - 2, target_s / max(t4, 1e-6))))
    b[...] = buf
    t0 = time.perf_counter()
    oracle.ltlt_colmajor(b, n, steps)
    dt = time.perf_counter() - t0
    flops = sum(float(n - k - 2) ** 2 for k in range(steps))
    return steps, dt, flops


def cpu_baseline(X, n, target_s):
    """The CPU oracle (plain scalar C, its rank-2 update split over OpenMP
    threads) on the first column steps of the same factorization, on every
    core this process is given, with a single-thread run beside it; nominal
    GFLOP/s with the n^3/3 convention (step k counts (n-k-2)^2 flops).  The
    first steps are the heaviest, so the rates are those of the large
    trailing sizes."""
    import numpy as np

    import oracle
    oracle.build()
    buf = np.ascontiguousarray(X.T)            # column-major image
    threads = oracle_threads()
    steps, dt, flops = _oracle_prefix_rate(buf, n, target_s, threads)
    s1, d1, f1 = _oracle_prefix_rate(buf, n, target_s / 2, 1)
    return {
        "value": flops / dt / 1e9,
        "unit": "GFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"first {steps} of {n - 2} column steps of the same n={n} input on {threads} threads "
                  f"({dt:.1f} s; nominal flops sum_k (n-k-2)^2 = {flops:.3e})",
        "single_thread": {"value": f1 / d1 / 1e9, "cores": 1,
                          "sample": f"first {s1} column steps, one thread ({d1:.1f} s)"},
        **host_info(),
    }


def run_cpu_oracle(args):
    """The whole oracle factorization + Pfaffian at --n on every core this
    process is given (no GPU involved): the full-size CPU baseline."""
    import numpy as np

    import oracle
    import synth
    oracle.build()
    gen = {"gauss": synth.skew_gauss, "graded": synth.skew_graded, "blockdiag4": synth.skew_blockdiag4}[args.input]
    np_dt = np.float64 if args.dtype == "f64" else np.float32
    n = args.n
    X = gen(n, args.seed).astype(np_dt)
    buf = np.ascontiguousarray(X.T)
    del X
    threads = oracle_threads()
    oracle.set_threads(threads)
    print(f"[cpu] oracle n={n} {args.dtype} on {threads} threads", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    ipiv = oracle.ltlt_colmajor(buf, n)
    packed = np.tril(buf.T, -1)
    logabs, sign = oracle.pfaffian_packed(packed, ipiv)
    dt = time.perf_counter() - t0
    out = {
        "metric": "CPU oracle LTL^T factorization + Pfaffian GFLOP/s (n^3/3)",
        "value": round(float(n) ** 3 / 3 / dt / 1e9, 3),
        "unit": "GFLOP/s",
        "seconds": round(dt, 2),
        "cores": threads,
        "dtype": args.dtype,
        "config": {"workload": f"whole oracle factorization of one n={n} {INPUT_TEXT[args.input]} matrix "
                               f"(seed {args.seed})", "n": n},
        "pfaffian": {"logabs": logabs, "sign": sign},
        **host_info(),
    }
    print(json.dumps(out), flush=True)


def launch_breakdown(lt, torch, step):
    """Per-kind milliseconds of one extra step, run after the timed region
    with every launch event-timed (the timed steps record the trailing
    updates only: each event record costs about 2 us of stream time)."""
    lt.profile_enable(True)
    step()
    torch.cuda.synchronize()
    lt.profile_enable(False)
    lt.device_status()
    return {k: round(v[1], 3) for k, v in lt.profile_read().items()}


INPUT_TEXT = {
    "gauss": "strict upper iid N(0,1)",
    "graded": "strict upper N(0,1) times 10^U(-3,3) per entry",
    "blockdiag4": "4x4 Gaussian skew-symmetric blocks on the diagonal",
}


# headers every kernel source includes; a kernel's code depends on them too
KERNEL_HEADERS = ("ltlt_device.h", "ltlt_internal.h")


def kernel_source_hash(source, headers=KERNEL_HEADERS):
    """sha256 of a kernel source followed by the shared headers it includes."""
    import hashlib
    h = hashlib.sha256()
    for name in (source, *headers):
        with open(os.path.join(ROOT, "paper_2005_06410_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(summary, source, headers=KERNEL_HEADERS):
    """HBM bytes per launch from a committed counter summary under profiles/
    (two rocprofv3 --pmc passes, FETCH_SIZE and WRITE_SIZE, scaled by a copy of
    known size), or None when the kernel's code (its source or the headers it
    includes) has changed since."""
    summ = os.path.join(ROOT, "profiles", summary)
    try:
        fields = {}
        for line in open(summ):
            if ":" in line and not line.startswith(("|", "#", " ", "-", "`")):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
        h = kernel_source_hash(source, headers)
        if not h.startswith(fields.get("source_sha256_prefix", "-")):
            return None
        return float(fields["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def conv_tensor_dev(a, torch):
    """numpy array (stored leftmost index fastest) -> GPU tensor, same layout."""
    import numpy as np
    a = np.asfortranarray(a)
    strides, acc = [], 1
    for d in a.shape:
        strides.append(acc)
        acc *= d
    flat = torch.from_numpy(np.ravel(a, order="F").copy()).to("cuda:0")
    return flat.as_strided(a.shape, tuple(strides))


def cpu_baseline_conv(specs, target_s):
    """The convolution oracle (direct loops of the paper's Figure 4 in scalar C,
    OpenMP over the batch index) on the same five layers at a batch of one
    entry per thread, repeated to about ``target_s`` seconds."""
    from oracle import conv as oc
    from synth import conv as sc
    threads = oracle_threads()
    oc.set_threads(threads)
    b = threads
    tensors = [sc.layer_tensors(sp, b, sc.layer_seed(sp)) for sp in specs]
    flops = 0.0
    reps = 0
    t0 = time.perf_counter()
    while True:
        for sp, (F, I) in zip(specs, tensors):
            O = oc.conv_direct(F, I, sp["s"], sp["p"])
            flops += 2.0 * O.size * sp["kh"] * sp["kw"] * sp["ci"]
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= target_s or reps >= 50:
            break
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"the five layers at batch {b} (one entry per thread), {reps} pass(es), {dt:.1f} s, "
                  f"fp64 sums of fp32 products",
        **host_info(),
    }


def run_convgemm(args):
    """The paper's own operator on MI355X: the five AlexNet convolution layers
    (Table 2) at batch b, each as one CONVGEMM launch on resident inputs.

    One step = the five layers in sequence.  The roofline is that of the
    dominant launch (layer 4, about half of the flops): algorithmic flops
    2 kn ho wo b kh kw ci per launch over its average HIP-event duration in
    the timed steps, against the fp32 matrix-core peak."""
    import torch

    import paper_2005_06410_amd as lt
    from synth import conv as sc
    b = args.conv_batch
    mt, nt = (int(v) for v in args.tile.split(","))
    stream = torch.cuda.current_stream(torch.device("cuda:0"))
    layers = []
    for sp in sc.ALEXNET_CONV:
        F, I = sc.layer_tensors(sp, b, sc.layer_seed(sp))
        ho = lt.conv_out_size(sp["hi"], sp["kh"], sp["s"], sp["p"])
        wo = lt.conv_out_size(sp["wi"], sp["kw"], sp["s"], sp["p"])
        kn = sp["kn"]
        O = torch.empty(kn * ho * wo * b, dtype=torch.float32, device="cuda:0").as_strided(
            (kn, ho, wo, b), (1, kn, kn * ho, kn * ho * wo))
        layers.append(dict(spec=sp, F=conv_tensor_dev(F, torch), I=conv_tensor_dev(I, torch), O=O,
                           flops=2.0 * kn * ho * wo * b * sp["kh"] * sp["kw"] * sp["ci"],
                           gemm=(kn, ho * wo * b, sp["kh"] * sp["kw"] * sp["ci"])))
        del F, I

    # a plain copy of known size (256 MiB read + 256 MiB written), untimed: the
    # calibration that the HBM counter passes of this workload are scaled by
    calib_src = torch.ones(64 << 20, dtype=torch.float32, device="cuda:0")
    calib_dst = torch.empty_like(calib_src)
    calib_dst.copy_(calib_src)
    del calib_src, calib_dst

    def step():
        evs = []
        for L in layers:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            lt.convgemm(L["F"], L["I"], L["spec"]["s"], L["spec"]["p"], out=L["O"], tile=(mt, nt),
                        path=args.conv_path)
            e1.record(stream)
            evs.append((e0, e1))
        return evs

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    all_evs = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    per_layer = [[a.elapsed_time(e) for a, e in (evs[i] for evs in all_evs)] for i in range(len(layers))]
    step_ms = [evs[0][0].elapsed_time(evs[-1][1]) for evs in all_evs]
    ms_step = sum(step_ms) / len(step_ms)
    total_flops = sum(L["flops"] for L in layers)
    value = total_flops / (ms_step * 1e-3) / 1e12
    dom = max(range(len(layers)), key=lambda i: layers[i]["flops"])
    dom_ms = sum(per_layer[dom]) / len(per_layer[dom])
    achieved = layers[dom]["flops"] / (dom_ms * 1e-3) / 1e12
    out = {
        "metric": f"CONVGEMM, AlexNet convolution layers (paper Table 2) at b={b}: fp32 TFLOP/s",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"the five AlexNet convolution layers of the paper's Table 2 (inputs 224x224x3 .. "
                        f"13x13x384, stride 4 then 1, no padding) at batch {b}, inputs U[0,1), He-Gaussian "
                        f"filters, each layer one implicit-im2col GEMM launch",
            "batch": b,
            "kernel": {0: "automatic", 1: "LDS-staged gather", 2: "register-direct"}[args.conv_path],
            "tile": "automatic" if (mt, nt) == (0, 0) else f"{mt}x{nt}",
            "parallelism": "single GPU",
        },
        "pct_of_peak": round(100.0 * value / FP32_PEAK_TF, 2),
        "roofline": {
            "kernel": f"convgemm_kernel, layer {layers[dom]['spec']['layer']} "
                      f"(GEMM {layers[dom]['gemm'][0]} x {layers[dom]['gemm'][1]} x {layers[dom]['gemm'][2]})",
            "bound": "mfma",
            "achieved": round(achieved, 3),
            "peak": FP32_PEAK_TF,
            "unit": "TFLOP/s",
            "frac": round(achieved / FP32_PEAK_TF, 4),
            "traffic": (measured_traffic("convgemm_alexnet_b80_f32.md", "convgemm.hip", headers=())
                        if (b, mt, nt, args.conv_path) == (80, 0, 0, 0) else None),
            "avg_launch_ms": round(dom_ms, 5),
        },
        "layers": [{"layer": L["spec"]["layer"], "gemm_mnk": L["gemm"],
                    "ms": round(sum(t) / len(t), 4),
                    "tflops": round(L["flops"] / (sum(t) / len(t) * 1e-3) / 1e12, 3)}
                   for L, t in zip(layers, per_layer)],
        "wall_s_timed_region": round(wall, 3),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_conv(sc.ALEXNET_CONV, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def run_batched(args):
    """Batched path: `batch` independent skew-symmetric matrices of order 64
    (contiguous, column-major), factored and their Pfaffians taken in one
    call.  HBM-bound: the algorithmic bytes are one read and one write of each
    strict lower triangle plus ipiv, log|Pf| and sign."""
    import numpy as np
    import torch

    import paper_2005_06410_amd as lt
    import synth

    n, batch = 64, args.batch
    np_dt = np.float64 if args.dtype == "f64" else np.float32
    Xs = synth.skew_batch(n, batch, 6 << 32)
    buf = np.stack([synth.to_colmajor(X) for X in Xs]).astype(np_dt)
    dev = torch.device("cuda:0")
    pristine = torch.from_numpy(buf.reshape(-1)).to(dev)
    work = torch.empty_like(pristine)
    A = work.as_strided((batch, n, n), (n * n, 1, n))
    ipiv = torch.empty((batch, n), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step():
        work.copy_(pristine)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        lt.factor_batched(A, ipiv=ipiv)
        e1.record(stream)
        return e0, e1

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in evs)
    ms_step = sum(ms) / len(ms)
    esz = 8 if args.dtype == "f64" else 4
    alg_bytes = batch * (2 * esz * n * (n - 1) / 2 + 4 * n + 8 + 4)
    gbs = alg_bytes / (ms_step * 1e-3) / 1e9
    out = {
        "metric": "batched LTL^T + Pfaffian, 8192 x n=64: GB/s of algorithmic HBM bytes",
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{batch} independent skew-symmetric n=64 {args.dtype} matrices, strict upper iid N(0,1) "
                        "(per-matrix seeds), factors + Pfaffians",
            "n": n,
            "batch": batch,
        },
        "roofline": {
            "kernel": "batched_kernel",
            "bound": "hbm",
            "achieved": round(gbs, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4),
            "traffic": (measured_traffic("batched_kernel_8192x64_f64.md", "ltlt_batched.hip")
                        if args.dtype == "f64" and batch == 8192 else None),
            "algorithmic_bytes": alg_bytes,
        },
        "nominal_gflops": round(batch * n ** 3 / 3.0 / (ms_step * 1e-3) / 1e9, 2),
    }
    print(json.dumps(out), flush=True)


def cpu_baseline_direct(X, n, target_s):
    """Time the CPU oracle's Pfaffian by the even column steps (scalar C, its
    rank-2 update split over the OpenMP threads this process is given) on its
    first steps; extrapolate by work (step k updates (n-k-2)^2 / 2 entries) to
    the whole Pfaffian and report the same effective n^3/3 GFLOP/s as the GPU
    line."""
    import numpy as np

    import oracle
    oracle.build()
    threads = oracle_threads()
    oracle.set_threads(threads)
    buf = np.ascontiguousarray(X.T)
    b1 = buf.copy()
    t0 = time.perf_counter()
    oracle.pfaffian_direct_colmajor(b1, n, 1)
    t1 = time.perf_counter() - t0
    del b1
    half = n // 2
    steps = int(max(1, min(half, target_s / max(t1, 1e-6))))
    t0 = time.perf_counter()
    oracle.pfaffian_direct_colmajor(buf, n, steps)
    dt = time.perf_counter() - t0
    work = lambda ks: sum(float(n - k - 2) ** 2 for k in ks)
    w_sample = work(range(0, 2 * steps, 2))
    w_total = work(range(0, n - 1, 2))
    t_total = dt * w_total / w_sample
    return {
        "value": float(n) ** 3 / 3.0 / t_total / 1e9,
        "unit": "GFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"first {steps} of {half} even column steps of the same n={n} input on {threads} threads "
                  f"({dt:.1f} s), extrapolated by work sum_k (n-k-2)^2 to {t_total:.0f} s per Pfaffian",
        **host_info(),
    }


def run_pfaffian(args):
    """Pfaffian by the even column steps only (ltlt_pfaffian_direct) of the
    headline matrix: half the pivot agreements of the factorization, the same
    trailing-update work.  Reported as effective GFLOP/s with the
    factorization's n^3/3 count, so the two lines compare directly."""
    import numpy as np
    import torch

    import paper_2005_06410_amd as lt
    import synth

    dev = torch.device("cuda:0")
    n, nb = args.n, args.nb
    np_dt = np.float64 if args.dtype == "f64" else np.float32
    X = synth.skew_gauss(n, args.seed).astype(np_dt)
    pristine = torch.from_numpy(synth.to_colmajor(X).ravel()).to(dev)
    work = torch.empty_like(pristine)
    A = work.as_strided((n, n), (1, n))
    ipiv = torch.empty(n, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step():
        work.copy_(pristine)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        _, logabs, sign = lt.pfaffian_direct(A, nb=nb, ipiv=ipiv)
        e1.record(stream)
        return e0, e1, logabs, sign

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    lt.device_status()
    lt.profile_enable("update")
    torch.cuda.synchronize()
    evs = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    lt.profile_enable(False)
    lt.device_status()
    prof = lt.profile_read()
    breakdown = launch_breakdown(lt, torch, step)
    ms_step = sum(a.elapsed_time(b) for a, b, _, _ in evs) / len(evs)
    peak_tf = FP64_PEAK_TF if args.dtype == "f64" else FP32_PEAK_TF
    gflops = float(n) ** 3 / 3.0 / (ms_step * 1e-3) / 1e9
    up_launches, up_ms, up_flops = prof["update"]
    achieved_tf = up_flops / (up_ms * 1e-3) / 1e12 if up_ms > 0 else 0.0
    out = {
        "metric": f"Pfaffian of one dense skew-symmetric n={n} {args.dtype} matrix by the even column steps: "
                  "effective GFLOP/s (n^3/3 per Pfaffian)",
        "value": round(gflops, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"Pfaffian of one dense skew-symmetric n={n} {args.dtype} matrix, strict upper iid N(0,1) "
                        f"(seed {args.seed}), even column steps only, {nb} columns per block",
            "n": n,
            "nb": nb,
            "parallelism": "single GPU",
        },
        "pct_of_peak": round(100.0 * gflops / (peak_tf * 1e3), 2),
        "roofline": {
            "kernel": "update_kernel (trailing update)",
            "bound": "mfma",
            "achieved": round(achieved_tf, 3),
            "peak": peak_tf,
            "unit": "TFLOP/s",
            "frac": round(achieved_tf / peak_tf, 4),
            "traffic": None,
            "launches_per_step": up_launches // max(args.steps, 1),
            "avg_launch_ms": round(up_ms / max(up_launches, 1), 5),
        },
        "breakdown_ms_per_step": breakdown,   # one extra step, every launch timed
        "pfaffian": {"logabs": float(evs[-1][2].item()), "sign": int(evs[-1][3].item())},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_direct(X, n, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def run_solve(args):
    """Solve X x = b with the factors of the headline matrix (ltlt_solve):
    factor once (untimed), then time the solve of nrhs right-hand sides.
    HBM-bound for few right-hand sides: the algorithmic bytes are two reads
    of the strict lower triangle of L (forward and backward substitution)
    plus one read and one write of B."""
    import numpy as np
    import torch

    import paper_2005_06410_amd as lt
    import synth

    dev = torch.device("cuda:0")
    n, nb, nrhs = args.n, args.nb, args.nrhs
    np_dt = np.float64 if args.dtype == "f64" else np.float32
    X = synth.skew_gauss(n, args.seed).astype(np_dt)
    flat = torch.from_numpy(synth.to_colmajor(X).ravel()).to(dev)
    A = flat.as_strided((n, n), (1, n))
    ipiv = lt.factor(A, nb=nb)
    rhs = synth.rng_for(args.seed + 1).standard_normal((n, nrhs)).astype(np_dt)
    b0 = torch.from_numpy(np.asfortranarray(rhs)).to(dev).t().contiguous().t()
    B = b0.clone().t().contiguous().t()
    stream = torch.cuda.current_stream(dev)

    def step():
        B.copy_(b0)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        lt.solve(A, ipiv, B)
        e1.record(stream)
        return e0, e1

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    lt.device_status()
    evs = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    lt.device_status()
    ms_step = sum(a.elapsed_time(b) for a, b in evs) / len(evs)
    esz = 8 if args.dtype == "f64" else 4
    alg_bytes = 2 * esz * n * (n - 1) / 2 + 2 * esz * n * nrhs + 4 * n
    gbs = alg_bytes / (ms_step * 1e-3) / 1e9
    out = {
        "metric": f"solve X x = b with the LTL^T factors, n={n} {args.dtype}, {nrhs} right-hand side(s): "
                  "GB/s of algorithmic HBM bytes",
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"x = X^-1 b from the factors of one dense skew-symmetric n={n} {args.dtype} matrix "
                        f"(strict upper iid N(0,1), seed {args.seed}), {nrhs} Gaussian right-hand side(s)",
            "n": n,
            "nrhs": nrhs,
            "parallelism": "single GPU",
        },
        "roofline": {
            "kernel": "solve_tri_kernel (forward + backward substitution)",
            "bound": "hbm",
            "achieved": round(gbs, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4),
            "traffic": None,
            "algorithmic_bytes": alg_bytes,
        },
    }
    if not args.no_cpu_baseline:
        import oracle
        from threadpoolctl import threadpool_limits
        packed = np.tril(flat.cpu().numpy().reshape(n, n).T, -1)
        piv = ipiv.cpu().numpy()
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            oracle.solve(packed, piv, rhs)
            dt = time.perf_counter() - t0
        out["cpu_baseline"] = {
            "value": round(alg_bytes / dt / 1e9, 4),
            "unit": "GB/s",
            "cores": 1,
            "kind": "oracle",
            "sample": f"one full solve of the same system ({dt:.1f} s, one BLAS thread; includes the oracle's "
                      "unpacking of L and T)",
        }
    print(json.dumps(out), flush=True)


def cpu_baseline_complex(X, n, target_s):
    """Time the CPU oracle's complex reduction (single-threaded scalar C) on
    its first column steps and report GFLOP/s with the complex convention of
    the GPU line: step k counts 4 (n-k-2)^2 real flops."""
    import numpy as np

    import oracle
    oracle.build()
    buf = np.ascontiguousarray(X.T)
    b1 = buf.copy()
    t0 = time.perf_counter()
    oracle.ltlt_colmajor(b1, n, 1)
    t1 = time.perf_counter() - t0
    del b1
    steps = int(max(1, min(n - 2, target_s / max(t1, 1e-6))))
    t0 = time.perf_counter()
    oracle.ltlt_colmajor(buf, n, steps)
    dt = time.perf_counter() - t0
    flops = sum(4.0 * float(n - k - 2) ** 2 for k in range(steps))
    return {
        "value": flops / dt / 1e9,
        "unit": "GFLOP/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"first {steps} of {n - 2} column steps of the same complex n={n} input, one thread "
                  f"(the complex oracle is not threaded) ({dt:.1f} s; nominal flops sum_k 4 (n-k-2)^2 = "
                  f"{flops:.3e})",
        **host_info(),
    }


def run_complex(args):
    """Factorization + Pfaffian of one dense complex skew-symmetric matrix
    (X^T = -X): the complex panel and, per block, the two real plane updates
    of depth 2(nb+1).  Reported as GFLOP/s of real flops, 4 n^3 / 3 per
    factorization (a complex multiply-add is four real ones)."""
    import numpy as np
    import torch

    import paper_2005_06410_amd as lt
    import synth

    dev = torch.device("cuda:0")
    n = args.n
    nb = args.nb if args.nb is not None else 128
    np_dt = np.complex128 if args.dtype == "f64" else np.complex64
    name = "c128" if args.dtype == "f64" else "c64"
    X = synth.skew_gauss_complex(n, args.seed, np_dt)
    pristine = torch.from_numpy(synth.to_colmajor(X).ravel()).to(dev)
    work = torch.empty_like(pristine)
    A = work.as_strided((n, n), (1, n))
    ipiv = torch.empty(n, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step():
        work.copy_(pristine)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        lt.factor(A, ipiv=ipiv, nb=nb)
        logabs, phase = lt.pfaffian(A, ipiv)
        e1.record(stream)
        return e0, e1, logabs, phase

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    lt.device_status()
    lt.profile_enable("update")
    torch.cuda.synchronize()
    evs = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    lt.profile_enable(False)
    lt.device_status()
    prof = lt.profile_read()
    breakdown = launch_breakdown(lt, torch, step)
    ms_step = sum(a.elapsed_time(b) for a, b, _, _ in evs) / len(evs)
    peak_tf = FP64_PEAK_TF if args.dtype == "f64" else FP32_PEAK_TF
    gflops = 4.0 * float(n) ** 3 / 3.0 / (ms_step * 1e-3) / 1e9
    up_launches, up_ms, up_flops = prof["update"]
    achieved_tf = up_flops / (up_ms * 1e-3) / 1e12 if up_ms > 0 else 0.0
    out = {
        "metric": f"complex LTL^T factorization GFLOP/s (4 n^3/3 real flops) at n={n} {name}",
        "value": round(gflops, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": name,
        "data": "synthetic",
        "config": {
            "workload": f"factorization + Pfaffian of one dense complex skew-symmetric n={n} {name} matrix, "
                        f"strict upper real and imaginary parts iid N(0,1) (seed {args.seed}), {nb} columns per block",
            "n": n,
            "nb": nb,
            "parallelism": "single GPU",
        },
        "pct_of_peak": round(100.0 * gflops / (peak_tf * 1e3), 2),
        "roofline": {
            "kernel": "update_kernel (trailing update, two real planes per block)",
            "bound": "mfma",
            "achieved": round(achieved_tf, 3),
            "peak": peak_tf,
            "unit": "TFLOP/s",
            "frac": round(achieved_tf / peak_tf, 4),
            "traffic": None,
            "launches_per_step": up_launches // max(args.steps, 1),
            "avg_launch_ms": round(up_ms / max(up_launches, 1), 5),
        },
        "breakdown_ms_per_step": breakdown,   # one extra step, every launch timed
        "pfaffian": {"logabs": float(evs[-1][2].item()), "phase": [float(v) for v in
                                                                 torch.view_as_real(evs[-1][3]).cpu().ravel()]},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_complex(X, n, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.nb is None and args.workload != "complex":
        args.nb = 128
    if args.gpus != 1:
        print(f"bench.py: runs on one GPU only (asked for --gpus {args.gpus}); "
              "the single-matrix factorization is not sharded across GPUs", file=sys.stderr)
        sys.exit(2)
    if args.workload == "cpu-oracle":
        run_cpu_oracle(args)
        return

    import numpy as np
    import torch

    import paper_2005_06410_amd as lt
    import synth

    if not os.path.exists(lt.LIB_PATH):
        from paper_2005_06410_amd import build as ltbuild
        ltbuild.build()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.workload == "batched":
        run_batched(args)
        return
    if args.workload == "pfaffian":
        run_pfaffian(args)
        return
    if args.workload == "solve":
        run_solve(args)
        return
    if args.workload == "complex":
        run_complex(args)
        return
    if args.workload == "convgemm":
        run_convgemm(args)
        return
    dev = torch.device("cuda:0")
    n, nb = args.n, args.nb
    np_dt = np.float64 if args.dtype == "f64" else np.float32
    t_dt = torch.float64 if args.dtype == "f64" else torch.float32

    gen = {"gauss": synth.skew_gauss, "graded": synth.skew_graded, "blockdiag4": synth.skew_blockdiag4}[args.input]
    X = gen(n, args.seed).astype(np_dt)
    buf = synth.to_colmajor(X)                        # (n, n): buf[c, i] = X[i, c]
    pristine = torch.from_numpy(buf.ravel()).to(dev)
    del buf
    work = torch.empty_like(pristine)
    A = work.as_strided((n, n), (1, n))
    ipiv = torch.empty(n, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step_events():
        work.copy_(pristine)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        lt.factor(A, ipiv=ipiv, nb=nb)
        logabs, sign = lt.pfaffian(A, ipiv)
        e1.record(stream)
        return e0, e1, logabs, sign

    for _ in range(args.warmup):
        step_events()
    torch.cuda.synchronize()
    lt.device_status()
    # measured matrix-core ceiling of this device (register-only MFMA loop)
    loop_peak_tf = lt.mfma_probe(args.dtype)

    lt.profile_enable("update")
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    evs = [step_events() for _ in range(args.steps)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    lt.profile_enable(False)
    lt.device_status()            # sticky: raises if a wait of any timed step gave up
    prof = lt.profile_read()
    breakdown = launch_breakdown(lt, torch, step_events)
    ms = [a.elapsed_time(b) for a, b, _, _ in evs]
    logabs = float(evs[-1][2].item())
    sign = int(evs[-1][3].item())
    ms_step = sum(ms) / len(ms)

    flops = float(n) ** 3 / 3.0
    gflops = flops / (ms_step * 1e-3) / 1e9
    nb_eff = nb if nb is not None else 128
    peak_tf = FP64_PEAK_TF if args.dtype == "f64" else FP32_PEAK_TF

    # dominant kernel: the trailing update.  Algorithmic flops per launch =
    # m2^2 * nb (the block's share of the n^3/3 count); achieved = their sum
    # over the timed launches / the summed launch durations.
    up_launches, up_ms, up_flops = prof["update"]
    achieved_tf = up_flops / (up_ms * 1e-3) / 1e12 if up_ms > 0 else 0.0

    out = {
        "metric": "LTL^T factorization GFLOP/s (n^3/3) at n=16384 fp64; % of FP64 MFMA peak",
        "value": round(gflops, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"one dense skew-symmetric n={n} {args.dtype} matrix, {INPUT_TEXT[args.input]} "
                        f"(seed {args.seed}), blocked LTL^T with panel width {nb_eff}, plus Pfaffian",
            "n": n,
            "nb": nb_eff,
            "input": args.input,
            "parallelism": "single GPU",
        },
        "pct_of_peak": round(100.0 * gflops / (peak_tf * 1e3), 2),
        "roofline": {
            "kernel": "update_kernel (trailing update)",
            "bound": "mfma",
            "achieved": round(achieved_tf, 3),
            "peak": peak_tf,
            "unit": "TFLOP/s",
            "frac": round(achieved_tf / peak_tf, 4),
            "measured_loop_peak": round(loop_peak_tf, 2),
            "frac_of_measured_loop_peak": round(achieved_tf / loop_peak_tf, 4) if loop_peak_tf > 0 else None,
            # counter passes exist for the headline workload only
            "traffic": (measured_traffic("update_kernel_hbm_traffic_n16384_f64_nb128.md", "ltlt_update.hip")
                        if (n, nb_eff, args.dtype, args.input) == (16384, 128, "f64", "gauss") else None),
            "launches_per_step": up_launches // max(args.steps, 1),
            "avg_launch_ms": round(up_ms / max(up_launches, 1), 5),
        },
        "breakdown_ms_per_step": breakdown,   # one extra step, every launch timed
        "wall_s_timed_region": round(wall, 3),
        "pfaffian": {"logabs": logabs, "sign": sign},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(X, n, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
