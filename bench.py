"""Throughput of the partial-straggler gradient-coding hot path on one MI355X.

One step is one pass of the whole hot path over one batch of synthetic input:
the chunk gradients of all N chunks (logistic regression, n samples each),
their sum (the exact target), the coefficient solves for every straggler
pattern, every simulated worker's encode, and the PS combine with the fused
squared error against the exact target.  Workload: m = N = 50 workers,
cyclic assignment with s = 4, d = 16384, n = 512, 10,000 straggler patterns
(20% full stragglers, the rest uniform partial progress), ell = 1.

    python bench.py [--steps K] [--warmup W] [--ell L] [--no-cpu-baseline]
                    [--no-configs] [--configs-full]

Prints one JSON line.  value = patterns decoded per second, whole job, with
every input resident in HBM before the timed region starts.  Outside the
step the same line carries the other workloads (`configs`): the latency of
a whole step of the two small ones, and for the m = 100 and m = 200 ones
every pattern (m = 100) or the first 1,000 patterns (m = 200) through
coefficients, encode and combine in batches, with their rooflines.  The
oracle's timing on this host's cores (`cpu_baseline`, `cpu_baseline_configs`)
runs first, before the GPU is touched.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "straggler patterns decoded/sec at m=50,d=16384; HBM GB/s and MFMA % of peak"
HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3
CPU_PROCS_MAX = 16           # worker processes of the oracle baseline: the machine's CPU share per GPU
LARGE_SUBSET = 1000          # m = 200 workload: patterns through encode and combine
BANDWIDTH_CPU_COLS = 1 << 15  # m = 100 workload: columns of the oracle's d-slice sample
LARGE_CPU_COLS = 1 << 14     # m = 200 workload: columns of the oracle's d-slice sample


def parse(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--ell", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", dest="configs", action="store_false",
                    help="skip the other workloads (reported under 'configs', outside the step)")
    ap.add_argument("--configs-full", action="store_true",
                    help="also run the m = 100 workload at ell = 8 and the m = 200 one at ell = 2 "
                         "and its least-squares run at ell = 1, 2, 4")
    ap.add_argument("--large-batch", type=int, default=0,
                    help="patterns per encode/combine call on the m = 200 workload (0: by ell)")
    ap.add_argument("--experiment", choices=["hotpath", "completion", "trigger", "ordering"],
                    default="hotpath",
                    help="hotpath: the headline step (default); completion: exact-GC completion times, "
                         "proposed vs original GC; trigger: error vs deadline, proposed vs original GC; "
                         "ordering: Algorithm 2 vs the best of 100 random orderings")
    ap.add_argument("--trials", type=int, default=1000)
    ap.add_argument("--mfma-points", type=int, default=256,
                    help="also time the chunk gradients at this many evaluation points (matrix-core "
                         "path; 0 = skip); reported under 'mfma', outside the step")
    ap.add_argument("--no-decode-large", dest="decode_large", action="store_false",
                    help="skip timing the coefficients of the 100,000-pattern m = 200 workload")
    ap.add_argument("--no-direct", dest="direct", action="store_false",
                    help="skip timing gc_decode_direct (reported under 'direct', outside the step)")
    ap.add_argument("--configs-only", choices=["given_m100_d1M", "given_m200_d16M_bf16", "decode_large"],
                    default=None,
                    help="profiling aid: run only this workload's configs (or the 100,000-pattern "
                         "coefficients) and print their JSON, without the headline step")
    ap.add_argument("--copy-probe-mib", type=int, default=1024,
                    help="size of a plain device copy run once before warm-up (counter calibration)")
    return ap.parse_args(argv)


def algorithmic_bytes(wl, ell, P, sent, esize=4):
    """Compulsory bytes per launch: every input read once, every output written once.
    ``sent`` = number of (pattern, worker) rows that transmit (psi > 0): only those
    rows of T are written by the encode and read by the combine.  ``esize`` = bytes per
    stored chunk-gradient value (4 fp32, 2 bf16)."""
    m, N, d, delta = wl.m, wl.N, wl.d, wl.delta
    L = -(-d // ell)
    enc = 4 * sent * L + esize * N * d + 4 * P * m + 4 * P * m * delta * ell + 4 * m * delta
    rec = 4 * sent * L + 4 * P * m + 4 * P * d + 4 * ell * m + 4 * d + 8 * P
    dcd = 4 * P * m + 4 * P * N + P + 4 * P + 4 * P * m * delta * ell + 4 * ell * m + 12 * N * delta
    grads = (4 * N * wl.n * wl.d + 4 * N * wl.n + 4 * d + 4 * N * d) if wl.n else 0
    return {"gc_encode": enc, "gc_reconstruct": rec, "gc_decode_coeffs": dcd, "gc_chunk_grads": grads,
            "gc_sum_chunks": esize * N * d + 4 * d}


def measured_traffic(wl, call, kernel_prefix=None):
    """HBM bytes per launch of the call's main kernel from the committed counter summary
    (profiles/hbm_traffic_<workload>.txt), or None when that kernel's sources have changed
    since the counters were taken (or no summary covers it)."""
    import hashlib
    prefix = kernel_prefix or {"gc_encode": "encode_kernel", "gc_reconstruct": "reconstruct_kernel"}[call]
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{wl.name}.txt")
    if not os.path.exists(path):
        return None
    data = None
    for line in open(path):
        if line.startswith("JSON "):
            data = json.loads(line[5:])
    if data is None:
        return None
    for name, k in data["kernels"].items():
        if name.startswith(prefix):
            h = hashlib.sha256()
            for src in k["sources"]:
                h.update(open(os.path.join(ROOT, src), "rb").read())
            return k["hbm_bytes"] if h.hexdigest()[:16] == k["sources_sha256_16"] else None
    return None


# ---------------------------------------------------------------------------
# the oracle on this host's cores (baseline only): a pool of forked worker processes, each
# single-threaded, over chunks and pattern windows; then one process pinned to one core.
# Runs before the GPU is touched, so the forks copy no GPU state.
# ---------------------------------------------------------------------------

_CPU = {}  # inputs the forked workers read (set in the parent before the pool starts)


def _log(msg):
    """Progress on stderr (the JSON line alone goes to stdout)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def _cpu_init(one_core):
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:  # pragma: no cover
        pass
    if one_core:
        os.sched_setaffinity(0, {min(os.sched_getaffinity(0))})


def _cpu_grads(i):
    import oracle.gradients as OG
    c = _CPU
    t0 = time.perf_counter()
    g = OG.chunk_gradient(c["X"][i], c["y"][i], c["w"], c["loss"])
    return i, g, time.perf_counter() - t0


def _cpu_given(i):
    from workloads import gen
    c = _CPU
    return i, gen.given_chunk(c["wl"], i, cols=c["cols"])


def _cpu_patterns(window):
    """Algorithm 1 (each worker's minimum-norm solve, with coverage and decodability),
    encode and combine for patterns lo..hi-1; CPU seconds per step."""
    import oracle.protocol as OP
    c = _CPU
    lo, hi = window
    O, psi, R, G, ell, d = c["O"], c["psi"], c["R"], c["G"], c["ell"], c["d"]
    t = np.zeros(3)
    for p in range(lo, hi):
        t0 = time.perf_counter()
        OP.coverage(O, psi[p])
        OP.decodable(O, psi[p], ell)
        OP.coef_err(O, psi[p], ell)
        B = OP.encoding_matrix(O, psi[p], R)
        t1 = time.perf_counter()
        T = OP.encode(B, G, ell)
        t2 = time.perf_counter()
        OP.reconstruct(T, R, d)
        t[0] += t1 - t0
        t[1] += t2 - t1
        t[2] += time.perf_counter() - t2
    return t


def _windows(P, parts):
    step = -(-P // parts)
    return [(lo, min(P, lo + step)) for lo in range(0, P, step)]


def _cpu_run(procs, one_core, fn, items):
    import multiprocessing as mp
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(procs, initializer=_cpu_init, initargs=(one_core,)) as pool:
        out = pool.map(fn, items, chunksize=1)
    return out, time.perf_counter() - t0


def cpu_oracle_config(wl, ell, procs, count=None, cols=None, one_core_count=0, grads=True):
    """Time the oracle on workload wl: chunk gradients of every chunk (regression workloads;
    given-gradient workloads generate theirs untimed), then Algorithm 1, encode and combine
    for the first ``count`` patterns (all by default), on ``procs`` worker processes and, for
    ``one_core_count`` patterns, on one core.  ``cols`` = a d-slice (given gradients only):
    times are scaled to the full d.  Returns per-step CPU seconds and wall times."""
    import oracle.assignment as OA
    import oracle.protocol as OP
    from workloads import gen
    P = wl.P if count is None else count
    _log(f"oracle on {procs} processes: {wl.name}, {P} patterns")
    O = OA.cyclic_O(wl.N, wl.m, wl.s)
    psi = gen.psi(wl, count=P)
    R = gen.shared_R(wl.m, ell).astype(np.float64)
    out = {"workload": wl.name, "ell": ell, "patterns": P, "procs": procs}
    t_grads_wall, t_grads_cpu = 0.0, 0.0
    _CPU.clear()
    if wl.n is not None:
        X, y, w = gen.regression_data(wl)
        _CPU.update(X=X, y=y, w=w, loss=wl.loss)
        res, t_grads_wall = _cpu_run(procs, False, _cpu_grads, range(wl.N))
        G = np.zeros((wl.N, wl.d))
        for i, g, dt in res:
            G[i] = g
            t_grads_cpu += dt
        d = wl.d
    else:
        _CPU.update(wl=wl, cols=cols)
        res, _ = _cpu_run(procs, False, _cpu_given, range(wl.N))
        Gs = np.stack([g for _, g in sorted(res, key=lambda r: r[0])])
        G = OP.widen(Gs, wl.g_dtype)
        d = G.shape[1]
    # on a d-slice the length-d steps (encode, combine) scale with d; the solves do not
    scale = np.array([1.0, wl.d / d, wl.d / d])
    _CPU.clear()
    _CPU.update(O=O, psi=psi, R=R, G=G, ell=ell, d=d)
    res, wall = _cpu_run(procs, False, _cpu_patterns, _windows(P, 4 * procs))
    steps = np.sum(res, axis=0) * scale
    out.update({
        "seconds_chunk_grads": t_grads_wall,
        "cpu_seconds": {"chunk_grads": t_grads_cpu, "decode_coeffs": float(steps[0]),
                        "encode": float(steps[1]), "reconstruct": float(steps[2])},
    })
    if cols is None:
        out.update({"wall_seconds_patterns": wall, "patterns_per_s": P / (t_grads_wall + wall),
                    "seconds_per_pattern": wall / P})
    else:
        # modelled: the per-pattern CPU time of the full d, spread over the worker processes
        cpu_pp = float(steps.sum()) / P
        out.update({"d_slice": f"{d} of {wl.d} columns; encode and combine times scaled by {wl.d / d:g}",
                    "seconds_per_pattern": cpu_pp / procs, "patterns_per_s": procs / cpu_pp,
                    "cpu_seconds_per_pattern": cpu_pp})
    if one_core_count:
        n1 = min(one_core_count, P)
        res, wall1 = _cpu_run(1, True, _cpu_patterns, [(0, n1)])
        t1 = res[0] * scale
        pp1 = float(t1.sum()) / n1 if cols is not None else wall1 / n1
        out["one_core"] = {"patterns": n1, "seconds_per_pattern": pp1, "patterns_per_s": 1.0 / pp1,
                           "cpu_seconds": dict(zip(("decode_coeffs", "encode", "reconstruct"),
                                                   (float(v) for v in t1)))}
        if wl.n is not None:
            # one-core chunk gradients: the same chunks, one after another
            _CPU.clear()
            _CPU.update(X=X, y=y, w=w, loss=wl.loss)
            r1, tg1 = _cpu_run(1, True, _cpu_grads, range(wl.N))
            out["one_core"]["seconds_chunk_grads"] = tg1
            out["one_core"]["step_patterns_per_s"] = P / (tg1 + P * pp1)
    _CPU.clear()
    return out


def cpu_baseline(args):
    """The oracle timed on this host (baseline only, not a target)."""
    from workloads import BANDWIDTH, HEADLINE, LARGE, SMALL, TINY
    host = len(os.sched_getaffinity(0))
    procs = min(CPU_PROCS_MAX, host)
    try:
        from threadpoolctl import threadpool_info
        blas = max([t.get("num_threads", 1) for t in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        blas = None
    head = cpu_oracle_config(HEADLINE, args.ell, procs, one_core_count=1500)
    base = {
        "value": head["patterns_per_s"], "unit": "patterns/s", "cores": procs, "kind": "oracle",
        "host_cores": host, "blas_threads_per_process": 1, "blas_threads_main": blas,
        "sample": (f"every pattern ({head['patterns']}) and every chunk gradient ({HEADLINE.N}) of "
                   f"the step, on {procs} single-threaded worker processes; one_core: "
                   f"{head['one_core']['patterns']} patterns and all chunk gradients on one core"),
        **{k: v for k, v in head.items() if k not in ("workload", "procs")},
    }
    others = {}
    if args.configs:
        others[TINY.name] = cpu_oracle_config(TINY, 1, procs)
        others[SMALL.name] = cpu_oracle_config(SMALL, 1, procs)
        for wl, cols in ((BANDWIDTH, BANDWIDTH_CPU_COLS), (LARGE, LARGE_CPU_COLS)):
            r = cpu_oracle_config(wl, 1, procs, count=procs, cols=slice(0, cols), one_core_count=2)
            r["sample"] = (f"the first {procs} patterns on the first {cols} columns, encode and combine "
                           f"times scaled to d = {wl.d}, as a per-pattern rate")
            others[wl.name] = r
    return base, others


# ---------------------------------------------------------------------------
# GPU timing
# ---------------------------------------------------------------------------

class Events:
    """HIP events on torch's current stream (the stream every gcx call is enqueued on)."""

    def __init__(self):
        import torch
        self.torch = torch
        self.ms = {}

    def time(self, name, fn):
        torch = self.torch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        out = fn()
        e1.record()
        self.pending = getattr(self, "pending", []) + [(name, e0, e1)]
        return out

    def collect(self):
        self.torch.cuda.synchronize()
        for name, e0, e1 in getattr(self, "pending", []):
            self.ms[name] = self.ms.get(name, 0.0) + e0.elapsed_time(e1)
        self.pending = []
        return self.ms


def time_many_points(gcx, wl, Xd, yd, b, dev, reps=5):
    """Chunk gradients of the same X at b evaluation points: two fp32 GEMMs per chunk on the
    matrix cores, 4 N n d b flops.  Reported against the fp32 MFMA peak."""
    import torch
    from workloads import gen
    W = torch.from_numpy(gen.eval_points(wl, b)).to(dev)
    G = torch.empty((b, wl.N, wl.d), dtype=torch.float32, device=dev)
    ws = torch.empty(gcx.gc_chunk_grads_workspace_size(wl.N, wl.n, wl.d, b), dtype=torch.uint8, device=dev)
    gcx.gc_chunk_grads(Xd, yd, W, gcx.GC_LOSS_LOGISTIC, G=G, workspace=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        gcx.gc_chunk_grads(Xd, yd, W, gcx.GC_LOSS_LOGISTIC, G=G, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    flops = 4.0 * wl.N * wl.n * wl.d * b
    tf = flops / (ms * 1e-3) / 1e12
    del G, ws, W
    torch.cuda.empty_cache()
    return {"bound": "mfma", "points": b, "ms": ms, "achieved": tf, "peak": FP32_MFMA_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": tf / FP32_MFMA_PEAK_TFLOPS, "dtype": "f32",
            "note": "gc_chunk_grads with W [b][d]: Z = X W^T, residuals, G = U^T X per chunk"}


def time_direct(gcx, wl, ell, G, gsum, psid, orderd, holderd, hposd, Rd, ghat, sqerr, reps=10):
    """gc_decode_direct on the step's own inputs: the same estimates and squared errors without
    the workers' transmitted vectors.  A dense fp32 contraction of the per-pattern mixing rows
    [P ell][N ell] with the block-split gradients [N ell][L]: 2 P ell N ell L flops, reported
    against the fp32 MFMA peak (time of the whole call: mixing matrices, contraction, error sums)."""
    import torch
    P = psid.shape[0]
    ws = torch.empty(gcx.gc_decode_direct_workspace_size(P, wl.N, wl.d, ell), dtype=torch.uint8,
                     device=G.device)

    def call():
        gcx.gc_decode_direct(G, psid, orderd, holderd, hposd, Rd, ghat=ghat, gsum=gsum, sqerr=sqerr,
                             workspace=ws)
    call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    L = -(-wl.d // ell)
    flops = 2.0 * P * ell * wl.N * ell * L
    tf = flops / (ms * 1e-3) / 1e12
    del ws
    return {"bound": "mfma", "ms": ms, "patterns_per_s": P / (ms * 1e-3), "achieved": tf,
            "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": tf / FP32_MFMA_PEAK_TFLOPS,
            "flops": flops, "dtype": "f32", "ghat": True,
            "note": "gc_decode_direct: estimate of every pattern from the chunk gradients through "
                    "M_i = R[:, S_i] pinv(R[:, S_i]), outside the step"}


def time_decode_large(gcx, psi, reps=10):
    """Coefficients for all 100,000 patterns of the m = 200, delta = 20 workload (exact run,
    ell = 1): the decode's bandwidth point, 1.6 GB of Bc written per call."""
    import torch
    from workloads import LARGE, gen
    wl = LARGE
    R = gen.shared_R(wl.m, 1)
    _, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_CYCLIC, wl.N, wl.m, wl.s)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    psid, od, hd, hpd, Rd = d(psi), d(order), d(holder), d(hpos), d(R)
    P = wl.P
    cov = torch.empty((P, wl.N), dtype=torch.int32, device="cuda")
    dec = torch.empty(P, dtype=torch.uint8, device="cuda")
    cerr = torch.empty(P, dtype=torch.int32, device="cuda")
    Bc = torch.empty((P, wl.m, wl.delta, 1), dtype=torch.float32, device="cuda")

    def call():
        gcx.gc_decode_coeffs(psid, od, hd, hpd, Rd, cov=cov, dec=dec, coef_err=cerr, Bc=Bc)
    call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    nbytes = algorithmic_bytes(wl, 1, P, 0)["gc_decode_coeffs"]
    gbs = nbytes / (ms * 1e-3) / 1e9
    out = {"workload": wl.name, "patterns": P, "ell": 1, "ms": ms, "patterns_per_s": P / (ms * 1e-3),
           "bound": "hbm", "algorithmic_bytes": nbytes, "achieved": gbs, "peak": HBM_PEAK_GBS,
           "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
           "decodable_frac": float((dec == 1).float().mean().item())}
    del cov, dec, cerr, Bc
    torch.cuda.empty_cache()
    return out


def small_config_latency(gcx, wl, ell, dev, reps=20):
    """A whole step (chunk gradients, their sum, coefficients, encode, combine with squared
    error) over every pattern of a small regression workload: latency per step."""
    import torch
    from workloads import gen
    X, y, w = gen.regression_data(wl)
    psi = gen.psi(wl)
    R = gen.shared_R(wl.m, ell)
    _, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_CYCLIC, wl.N, wl.m, wl.s)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    Xd, yd, wd, psid, Rd, od, hd, hpd = (t(a) for a in (X, y, w, psi, R, order, holder, hpos))
    P, L = wl.P, -(-wl.d // ell)
    G = torch.empty((wl.N, wl.d), device=dev)
    gsum = torch.empty(wl.d, device=dev)
    ws_g = torch.empty(gcx.gc_chunk_grads_workspace_size(wl.N, wl.n, wl.d, 1), dtype=torch.uint8, device=dev)
    cov = torch.empty((P, wl.N), dtype=torch.int32, device=dev)
    dec = torch.empty(P, dtype=torch.uint8, device=dev)
    cerr = torch.empty(P, dtype=torch.int32, device=dev)
    Bc = torch.empty((P, wl.m, wl.delta, ell), device=dev)
    T = torch.empty((P, wl.m, L), device=dev)
    ghat = torch.empty((P, wl.d), device=dev)
    sq = torch.empty(P, dtype=torch.float64, device=dev)
    ws_r = torch.empty(max(1, gcx.gc_reconstruct_workspace_size(P, wl.m, wl.d, ell)), dtype=torch.uint8,
                       device=dev)

    def step():
        gcx.gc_chunk_grads(Xd, yd, wd, 0 if wl.loss == "linear" else 1, G=G, workspace=ws_g)
        gcx.gc_sum_chunks(G, gsum=gsum)
        gcx.gc_decode_coeffs(psid, od, hd, hpd, Rd, cov=cov, dec=dec, coef_err=cerr, Bc=Bc)
        gcx.gc_encode(G, psid, od, Bc, T=T)
        gcx.gc_reconstruct(T, Rd, wl.d, psid, ghat=ghat, gsum=gsum, sqerr=sq, workspace=ws_r)
    for _ in range(3):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / reps
    return {"workload": wl.name, "ell": ell, "patterns": P, "ms_per_step": ms,
            "patterns_per_s": P / (ms * 1e-3),
            "decoded_gradients_per_s": float((dec == 1).sum().item()) / (ms * 1e-3),
            "note": "latency-bound (launch and small kernels); no roofline claim"}


def given_config(gcx, wl, ell, variant, psi, Gd, gsum, batch, dev):
    """Coefficients, encode and combine (with squared error) over the patterns ``psi`` of a
    given-gradient workload in batches of ``batch`` patterns per call; per-call HIP events.
    Returns rates, algorithmic bytes per call kind and roofline fractions."""
    import torch
    from workloads import gen
    P = len(psi)
    L = -(-wl.d // ell)
    esize = Gd.element_size()
    _, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_CYCLIC, wl.N, wl.m, wl.s)
    od, hd, hpd = (torch.from_numpy(a).to(dev) for a in (order, holder, hpos))
    Rd = torch.from_numpy(gen.shared_R(wl.m, ell)).to(dev)
    psid_all = torch.from_numpy(psi).to(dev)
    T = torch.empty((batch, wl.m, L), device=dev)
    ghat = torch.empty((batch, wl.d), device=dev)
    sq = torch.empty(P, dtype=torch.float64, device=dev)
    cov = torch.empty((batch, wl.N), dtype=torch.int32, device=dev)
    dec = torch.empty(P, dtype=torch.uint8, device=dev)
    cerr = torch.empty(batch, dtype=torch.int32, device=dev)
    Bc = torch.empty((batch, wl.m, wl.delta, ell), device=dev)
    ws = torch.empty(max(1, gcx.gc_reconstruct_workspace_size(batch, wl.m, wl.d, ell)), dtype=torch.uint8,
                     device=dev)

    _log(f"{wl.name} {variant} ell={ell}: {P} patterns, {batch} per call")

    def run(ev, lo, hi):
        n = hi - lo
        ps = psid_all[lo:hi]
        B, Tb = Bc[:n], T[:n]
        ev.time("gc_decode_coeffs", lambda: gcx.gc_decode_coeffs(ps, od, hd, hpd, Rd, cov=cov[:n],
                                                                  dec=dec[lo:hi], coef_err=cerr[:n], Bc=B))
        ev.time("gc_encode", lambda: gcx.gc_encode(Gd, ps, od, B, T=Tb))
        ev.time("gc_reconstruct", lambda: gcx.gc_reconstruct(Tb, Rd, wl.d, ps, ghat=ghat[:n], gsum=gsum,
                                                              sqerr=sq[lo:hi], workspace=ws))
    run(Events(), 0, min(batch, P))        # warm-up batch
    torch.cuda.synchronize()
    ev = Events()
    t0 = time.perf_counter()
    for lo in range(0, P, batch):
        run(ev, lo, min(P, lo + batch))
    ms = ev.collect()
    wall = time.perf_counter() - t0
    total_ms = sum(ms.values())
    sent = int((psi > 0).sum())
    calls = -(-P // batch)
    # per-call compulsory bytes summed over the calls: G is read once per encode call
    enc_b = 4 * sent * L + calls * esize * wl.N * wl.d + 4 * P * wl.m * (1 + wl.delta * ell)
    rec_b = 4 * sent * L + 4 * P * wl.m + 4 * P * wl.d + 8 * P + calls * (4 * ell * wl.m + 4 * wl.d)
    dcd_b = algorithmic_bytes(wl, ell, P, sent)["gc_decode_coeffs"]
    roof = {}
    for name, nb in (("gc_encode", enc_b), ("gc_reconstruct", rec_b), ("gc_decode_coeffs", dcd_b)):
        gbs = nb / (ms[name] * 1e-3) / 1e9
        roof[name] = {"ms": ms[name], "algorithmic_bytes": nb, "achieved": gbs, "frac": gbs / HBM_PEAK_GBS}
    decs = dec.cpu().numpy()
    out = {"workload": wl.name, "variant": variant, "ell": ell, "patterns": P, "patterns_per_call": batch,
           "g_dtype": wl.g_dtype, "transmitting_rows_frac": sent / (P * wl.m),
           "ms": total_ms, "wall_s": wall,
           "patterns_per_s": P / (total_ms * 1e-3),
           "decoded_gradients_per_s": float((decs == 1).sum()) / (total_ms * 1e-3),
           "decodable_frac": float((decs == 1).mean()),
           "bound": "hbm", "peak": HBM_PEAK_GBS, "unit": "GB/s", "kernels": roof,
           "mse_vs_sum_g": float(sq.mean().item() / wl.d)}
    del T, ghat, sq, cov, dec, cerr, Bc, ws
    torch.cuda.empty_cache()
    return out


def device_G(wl, dev, seed=0):
    """Chunk gradients [N][d] i.i.d. N(0, 1) drawn on the GPU from torch's seeded generator,
    stored fp32 or rounded to bf16 (the same distribution as the host generator the parity
    tests use; the values differ)."""
    import torch
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    G = torch.randn((wl.N, wl.d), generator=g, device=dev, dtype=torch.float32)
    return G.to(torch.bfloat16) if wl.g_dtype == "bf16" else G


def large_batch(ell, override):
    """Patterns per encode/combine call on the m = 200 workload (T is 13.4 GB per pattern at
    ell = 1): as many as keep T near 215 GB, so G's 6.7 GB are read once per 16 / 32 / 64
    patterns and the matrix-core encode gets 16 / 32 patterns per tile (measured: 16 patterns
    per call write T 20% faster than 8 at ell = 1)."""
    if override:
        return override
    return {1: 16, 2: 32, 4: 64}.get(ell, 16)


def run_configs(gcx, args, dev, psi_large, only=None):
    """The other workloads, outside the step (``only``: that one workload alone)."""
    import torch
    from workloads import BANDWIDTH, LARGE, SMALL, TINY, gen
    out = {}
    if only is None:
        for wl in (TINY, SMALL):
            _log(f"{wl.name}: whole-step latency")
            out[wl.name] = small_config_latency(gcx, wl, 1, dev)
    # m = 100, d = 2^20: all 10,000 patterns in batches
    if only in (None, BANDWIDTH.name):
        wl = BANDWIDTH
        Gd = device_G(wl, dev)
        gsum = gcx.gc_sum_chunks(Gd)
        psi = gen.psi(wl)
        rows = {}
        for ell in ((1, 2, 8) if args.configs_full else (1, 2)):
            batch = {1: 256, 2: 512, 8: 1024}[ell]
            rows[f"exact_l{ell}"] = given_config(gcx, wl, ell, "exact", psi, Gd, gsum, batch, dev)
        out[wl.name] = rows
        del Gd, gsum
        torch.cuda.empty_cache()
    if only not in (None, LARGE.name):
        return out
    # m = 200, d = 2^24, bf16: the first 1,000 patterns through encode and combine
    wl = LARGE
    Gd = device_G(wl, dev)
    gsum = gcx.gc_sum_chunks(Gd)
    rows = {}
    runs = [("exact", 1)]
    if args.configs_full:
        runs += [("exact", 2), ("ls", 1), ("ls", 2), ("ls", 4)]
    for variant, ell in runs:
        psi = psi_large[:LARGE_SUBSET] if variant == "exact" else gen.psi(wl, count=LARGE_SUBSET, variant="ls")
        rows[f"{variant}_l{ell}"] = given_config(gcx, wl, ell, variant, psi, Gd, gsum,
                                                  large_batch(ell, args.large_batch), dev)
    out[wl.name] = rows
    del Gd, gsum
    torch.cuda.empty_cache()
    return out


def _psi_window(window):
    from workloads import LARGE, gen
    lo, hi = window
    return gen.psi(LARGE, start=lo, count=hi - lo)


def large_patterns(procs):
    """The 100,000 exact-run patterns of the m = 200 workload, generated by window on the
    worker pool (identical to one gen.psi call)."""
    from workloads import LARGE
    res, _ = _cpu_run(procs, False, _psi_window, _windows(LARGE.P, 10 * procs))
    return np.concatenate(res)


def _tables(gcx, kind, m, nu):
    """Cyclic or regular-graph (Algorithm 2 in the library) assignment tables for m = N."""
    from workloads import gen
    if kind == "cyclic":
        return gcx.gc_assign(gcx.GC_ASSIGN_CYCLIC, m, m, nu - 1)
    A = gen.random_regular_graph(m, nu).astype(np.int32)
    return gcx.gc_assign(gcx.GC_ASSIGN_REGULAR, m, m, -1, A, nu, nu)


def experiment_completion(args):
    """Exact-GC completion time (Sec. 4): cyclic N = m = 200 with delta = 8, and a random
    8-regular graph; alpha = delta - ell failed workers; Exp(1) chunk times."""
    import torch

    from paper_2405_19509_amd import gcx
    from workloads import GRAPH, Workload, gen
    dev = torch.device("cuda:0")
    out = {"metric": "exact-GC completion time, proposed vs original GC (simulated time units)",
           "unit": "trials/s", "n_gpus": 1, "higher_is_better": True, "data": "synthetic",
           "config": {"workload": "completion_m200_delta8", "m": 200, "delta": 8, "trials": args.trials,
                      "failures": "delta - ell", "chunk_times": "Exp(1)"}, "results": {}}
    total_ms, total_trials = 0.0, 0
    for kind in ("cyclic", "graph"):
        O, order, holder, hpos = _tables(gcx, kind, 200, 8)
        hd, pd = torch.from_numpy(holder).to(dev), torch.from_numpy(hpos).to(dev)
        rows = {}
        for ell in range(1, 8):
            wl = Workload(name="c", N=200, m=200, s=7, d=1, P=1, ells=(ell,)) if kind == "cyclic" else GRAPH
            tau, failed = gen.chunk_times(wl, args.trials, seed=100 + ell, failed=8 - ell)
            taud, fd = torch.from_numpy(tau).to(dev), torch.from_numpy(failed.astype(np.uint8)).to(dev)
            gcx.gc_completion_times(taud, hd, pd, ell, failed=fd)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            part, orig = gcx.gc_completion_times(taud, hd, pd, ell, failed=fd)
            e1.record()
            torch.cuda.synchronize()
            total_ms += e0.elapsed_time(e1)
            total_trials += args.trials
            p, o = part.cpu().numpy(), orig.cpu().numpy()
            rows[str(ell)] = {"proposed_mean": float(p.mean()), "original_mean": float(o.mean()),
                              "proposed_std": float(p.std()), "original_std": float(o.std()),
                              "ratio": float(o.mean() / p.mean())}
        out["results"][kind] = rows
    out["value"] = total_trials / (total_ms * 1e-3)
    out["paper_context"] = ("Sec. 4: proposed protocol about 2x faster than original GC for exact recovery "
                            "(cyclic N = m = 200, delta = 8, and graph G1; alpha = delta - ell; Exp(1)); "
                            "original GC on G1 at ell = 1 about 6 time units")
    print(json.dumps(out))


def experiment_trigger(args):
    """Error vs deadline T on a random 8-regular graph (m = 200), alpha = 7 failures:
    the proposed protocol's coefficient error sum_i max(0, ell - Delta_i) (equal to its
    least-squares residual, Sec. 2.1) for ell = 1, 2, 3, and original GC's least-squares
    error over fully finished workers (ell = 1)."""
    import torch

    from paper_2405_19509_amd import gcx
    from workloads import GRAPH, gen
    dev = torch.device("cuda:0")
    O, order, holder, hpos = _tables(gcx, "graph", 200, 8)
    od, hd, pd = (torch.from_numpy(a).to(dev) for a in (order, holder, hpos))
    T = np.arange(0.0, 24.01, 1.0)
    tau, failed = gen.chunk_times(GRAPH, args.trials, seed=7)
    taud, fd, Td = (torch.from_numpy(a).to(dev) for a in (tau, failed.astype(np.uint8), T))
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    psi = gcx.gc_progress(taud, Td, failed=fd).reshape(-1, 200)
    curves = {}
    for ell in (1, 2, 3):
        _, _, cerr, _ = gcx.gc_decode_coeffs(psi, od, hd, pd, torch.from_numpy(gen.shared_R(200, ell)).to(dev),
                                             coverage_only=True)
        curves[f"proposed_ell{ell}"] = cerr
    err_o, iters = gcx.gc_original_ls(psi, od, hd)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    res = {k: v.view(args.trials, len(T)).double().mean(0).cpu().numpy().tolist() for k, v in curves.items()}
    res["original_ell1"] = err_o.view(args.trials, len(T)).mean(0).cpu().numpy().tolist()
    out = {"metric": "coefficient-space error vs deadline, proposed (ell=1,2,3) vs original GC (ell=1)",
           "unit": "(trial, deadline) patterns/s", "value": args.trials * len(T) / (ms * 1e-3), "n_gpus": 1,
           "higher_is_better": True, "data": "synthetic",
           "config": {"workload": "trigger_graph_m200_nu8", "m": 200, "nu": 8, "failures": 7,
                      "trials": args.trials, "deadlines": T.tolist()},
           "results": res, "max_cgls_iters": int(iters.max().item()),
           "paper_context": ("Sec. 4, Fig. 3(a): on G1 (m = 200, nu = 8, alpha = 7) the proposed protocol's "
                             "MSE is several orders of magnitude below original GC's as T grows, also for "
                             "ell >= 2; its estimate (ell - Delta)/ell per column tracks the error")}
    print(json.dumps(out))


def experiment_ordering(args):
    """Algorithm 2's ordering against the best (smallest Q_max) of 100 random orderings of the
    same random 8-regular support, m = 200 (the appendix comparison of Sec. 4): exact-GC
    completion time of the proposed protocol for ell = 1..7 (alpha = delta - ell failures), and
    its coefficient error vs deadline for ell = 1, 2, 3 (alpha = 7).  Both orderings see the
    same chunk times: entry [r][j][t] is the time worker j spends on its t-th chunk."""
    import torch

    from paper_2405_19509_amd import gcx
    from workloads import GRAPH, gen
    dev = torch.device("cuda:0")
    m, nu = GRAPH.m, GRAPH.delta
    A = gen.random_regular_graph(m, nu).astype(np.int32)
    O_opt, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_REGULAR, m, m, -1, A.copy(), nu, nu)
    cands = gen.random_orderings(A, 100)
    qs = [gcx.gc_qmax(O)[1] for O in cands]
    best = int(np.argmin(qs))
    _, order_r, holder_r, hpos_r = gcx.gc_assign(gcx.GC_ASSIGN_ORDER, m, m, -1, cands[best].copy(), nu, nu)
    tabs = {"optimal": (order, holder, hpos), "random_best_of_100": (order_r, holder_r, hpos_r)}
    tabs = {k: tuple(torch.from_numpy(a).to(dev) for a in v) for k, v in tabs.items()}
    out = {"metric": "Algorithm 2 ordering vs best-of-100 random ordering (Q_max), proposed protocol",
           "unit": "trials/s", "n_gpus": 1, "higher_is_better": True, "data": "synthetic",
           "config": {"workload": "ordering_graph_m200_nu8", "m": m, "nu": nu, "trials": args.trials},
           "q_max": {"optimal": gcx.gc_qmax(O_opt)[1], "random_best_of_100": qs[best],
                     "random_median_of_100": float(np.median(qs))},
           "completion": {}, "error_vs_deadline": {}}
    total_ms, total = 0.0, 0
    for ell in range(1, nu):
        tau, failed = gen.chunk_times(GRAPH, args.trials, seed=100 + ell, failed=nu - ell)
        taud, fd = torch.from_numpy(tau).to(dev), torch.from_numpy(failed.astype(np.uint8)).to(dev)
        row = {}
        for name, (od, hd, pd) in tabs.items():
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            part, _ = gcx.gc_completion_times(taud, hd, pd, ell, failed=fd)
            e1.record()
            torch.cuda.synchronize()
            total_ms += e0.elapsed_time(e1)
            total += args.trials
            p = part.cpu().numpy()
            row[name] = {"mean": float(p.mean()), "std": float(p.std())}
        out["completion"][str(ell)] = row
    T = np.arange(0.0, 16.01, 1.0)
    tau, failed = gen.chunk_times(GRAPH, args.trials, seed=7)
    taud, fd, Td = (torch.from_numpy(a).to(dev) for a in (tau, failed.astype(np.uint8), T))
    psi = gcx.gc_progress(taud, Td, failed=fd).reshape(-1, m)
    for name, (od, hd, pd) in tabs.items():
        curves = {}
        for ell in (1, 2, 3):
            _, _, cerr, _ = gcx.gc_decode_coeffs(psi, od, hd, pd, torch.from_numpy(gen.shared_R(m, ell)).to(dev),
                                                 coverage_only=True)
            curves[f"ell{ell}"] = cerr.view(args.trials, len(T)).double().mean(0).cpu().numpy().tolist()
        out["error_vs_deadline"][name] = curves
    out["deadlines"] = T.tolist()
    out["value"] = total / (total_ms * 1e-3)
    out["paper_context"] = ("Appendix of Sec. 4: on G1 the optimal ordering has lower completion time and "
                            "lower MSE than the best of 100 random orderings (by Q_max), the MSE by orders "
                            "of magnitude at some deadlines")
    print(json.dumps(out))


def configs_only(args):
    """One workload's configs (or the 100,000-pattern coefficients) alone, for traces and
    counters per workload; prints their JSON (not the bench line)."""
    # patterns generated in this process: under a profiler, forked workers can hang in the
    # profiler's own teardown
    from workloads import LARGE, gen
    large = args.configs_only in ("given_m200_d16M_bf16", "decode_large")
    psi_large = gen.psi(LARGE) if large else None
    import torch

    from paper_2405_19509_amd import gcx
    gcx.load()  # fail loudly if the HIP library is missing
    assert torch.cuda.is_available(), "bench.py needs the GPU"
    dev = torch.device("cuda:0")
    if args.configs_only == "decode_large":
        out = {"decode_large": time_decode_large(gcx, psi_large)}
    else:
        out = {"configs": run_configs(gcx, args, dev, psi_large, only=args.configs_only)}
    print(json.dumps(out))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (the hot path is one GPU's share; got --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    if args.experiment == "completion":
        return experiment_completion(args)
    if args.experiment == "trigger":
        return experiment_trigger(args)
    if args.experiment == "ordering":
        return experiment_ordering(args)
    if args.configs_only:
        return configs_only(args)

    # ---- host work first, before the GPU is touched: the oracle baseline and the
    # 100,000 patterns of the m = 200 workload, both on forked worker processes ----
    procs = min(CPU_PROCS_MAX, len(os.sched_getaffinity(0)))
    cpu_base, cpu_configs = (None, None) if args.no_cpu_baseline else cpu_baseline(args)
    psi_large = large_patterns(procs) if (args.decode_large or args.configs) else None

    import torch

    from paper_2405_19509_amd import gcx
    from workloads import HEADLINE, gen

    gcx.load()  # fail loudly if the HIP library is missing
    assert torch.cuda.is_available(), "bench.py needs the GPU"
    wl, ell, P = HEADLINE, args.ell, HEADLINE.P
    dev = torch.device("cuda:0")

    # ---- inputs (host generation, then resident in HBM) ----
    X, y, w = gen.regression_data(wl)
    psi = gen.psi(wl)
    R = gen.shared_R(wl.m, ell)
    O, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_CYCLIC, wl.N, wl.m, wl.s)

    def d(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    Xd, yd, wd, psid, Rd = d(X), d(y), d(w), d(psi), d(R)
    orderd, holderd, hposd = d(order), d(holder), d(hpos)
    L = -(-wl.d // ell)
    G = torch.empty((wl.N, wl.d), dtype=torch.float32, device=dev)
    gsum = torch.empty(wl.d, dtype=torch.float32, device=dev)
    ws_g = torch.empty(gcx.gc_chunk_grads_workspace_size(wl.N, wl.n, wl.d, 1), dtype=torch.uint8, device=dev)
    cov = torch.empty((P, wl.N), dtype=torch.int32, device=dev)
    dec = torch.empty(P, dtype=torch.uint8, device=dev)
    cerr = torch.empty(P, dtype=torch.int32, device=dev)
    Bc = torch.empty((P, wl.m, wl.delta, ell), dtype=torch.float32, device=dev)
    T = torch.empty((P, wl.m, L), dtype=torch.float32, device=dev)
    ghat = torch.empty((P, wl.d), dtype=torch.float32, device=dev)
    sqerr = torch.empty(P, dtype=torch.float64, device=dev)
    ws_r = torch.empty(max(1, gcx.gc_reconstruct_workspace_size(P, wl.m, wl.d, ell)), dtype=torch.uint8,
                       device=dev)
    torch.cuda.synchronize()

    names = ["gc_chunk_grads", "gc_sum_chunks", "gc_decode_coeffs", "gc_encode", "gc_reconstruct"]

    def step(ev=None):
        def mark(i):
            if ev is not None:
                ev[i].record()
        mark(0)
        gcx.gc_chunk_grads(Xd, yd, wd, gcx.GC_LOSS_LOGISTIC, G=G, workspace=ws_g)
        mark(1)
        gcx.gc_sum_chunks(G, gsum=gsum)
        mark(2)
        gcx.gc_decode_coeffs(psid, orderd, holderd, hposd, Rd, cov=cov, dec=dec, coef_err=cerr, Bc=Bc)
        mark(3)
        gcx.gc_encode(G, psid, orderd, Bc, T=T)
        mark(4)
        gcx.gc_reconstruct(T, Rd, wl.d, psid, ghat=ghat, gsum=gsum, sqerr=sqerr, workspace=ws_r)
        mark(5)

    # a plain copy of known size, for calibrating HBM byte counters
    if args.copy_probe_mib > 0:
        nb = args.copy_probe_mib << 20
        src = torch.empty(nb // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    _log(f"headline step: {args.warmup} warm-up + {args.steps} timed")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # ---- timed region: exactly K steps ----
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    per = {n: [] for n in names}
    for ev in evs:
        for i, n in enumerate(names):
            per[n].append(ev[i].elapsed_time(ev[i + 1]))
    avg_ms = {n: float(np.mean(v)) for n, v in per.items()}
    ms_per_step = elapsed * 1e3 / args.steps
    value = P * args.steps / elapsed

    sent = int((psi > 0).sum())
    nbytes = algorithmic_bytes(wl, ell, P, sent)
    dominant = max(("gc_encode", "gc_reconstruct"), key=lambda n: avg_ms[n])
    achieved = nbytes[dominant] / (avg_ms[dominant] * 1e-3) / 1e9
    gbs = {n: nbytes[n] / (avg_ms[n] * 1e-3) / 1e9 for n in names}

    decs = dec.cpu().numpy()
    se = sqerr.cpu().numpy()
    out = {
        "metric": METRIC, "value": value, "unit": "patterns/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": wl.name, "N": wl.N, "m": wl.m, "s": wl.s, "d": wl.d, "n": wl.n,
                   "loss": wl.loss, "patterns": P, "ell": ell, "assignment": "cyclic",
                   "stragglers": "10 full + uniform partial progress",
                   "transmitting_rows_frac": sent / (P * wl.m)},
        "roofline": {"bound": "hbm", "kernel": dominant, "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic(wl, dominant) if ell == 1 else None,
                     "algorithmic_bytes": nbytes[dominant], "avg_ms": avg_ms[dominant]},
        "kernels_ms": avg_ms,
        "kernels_gbs": gbs,
        "decoded_gradients_per_s": float((decs == 1).sum()) * args.steps / elapsed,
        "coefficient_patterns_per_s": P / (avg_ms["gc_decode_coeffs"] * 1e-3),
        "quality": {"decodable_frac": float((decs == 1).mean()),
                    "mean_coef_err": float(cerr.float().mean().item()),
                    "mse_vs_sum_g": float(se.mean() / wl.d),
                    "mse_decodable": float(se[decs == 1].mean() / wl.d) if (decs == 1).any() else None},
    }
    if args.direct:
        out["direct"] = time_direct(gcx, wl, ell, G, gsum, psid, orderd, holderd, hposd, Rd, ghat, sqerr)
        # both routes give the same squared errors (up to fp32 rounding of the estimates)
        se_d = sqerr.cpu().numpy()
        out["direct"]["sqerr_max_abs_diff_vs_step"] = float(np.abs(np.sqrt(se_d) - np.sqrt(se)).max())
    del T, ghat, Bc, cov, ws_r
    torch.cuda.empty_cache()
    if args.mfma_points > 0:
        out["mfma"] = time_many_points(gcx, wl, Xd, yd, args.mfma_points, dev)
        if args.mfma_points != 64:
            out["mfma_b64"] = time_many_points(gcx, wl, Xd, yd, 64, dev)
    del Xd, G
    torch.cuda.empty_cache()
    if args.decode_large:
        _log("coefficients of the 100,000-pattern m = 200 workload")
        out["decode_large"] = time_decode_large(gcx, psi_large)
    if args.configs:
        out["configs"] = run_configs(gcx, args, dev, psi_large)
    if cpu_base is not None:
        out["cpu_baseline"] = cpu_base
        if cpu_configs:
            out["cpu_baseline_configs"] = cpu_configs
    print(json.dumps(out))


if __name__ == "__main__":
    main()
