"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

Every quantity draws from its own child of ``numpy.random.SeedSequence(seed)``
so that changing one size never changes another quantity's values:

    spawn key (0, i)   chunk i of X, or chunk gradient i when gradients are given
    spawn key (1,)     w*  (the model generating the labels)
    spawn key (2,)     label noise / Bernoulli draws
    spawn key (3,)     w   (the evaluation point)
    spawn key (4,)     R   (the shared ell x m Gaussian matrix)
    spawn key (5, 0)   per-worker speed factors (heterogeneous model)
    spawn key (5, 1+b) straggler patterns of batch b (PATTERN_BATCH patterns)
    spawn key (6, m, nu) random nu-regular graphs on m vertices (regular-graph assignments)
    spawn key (7, trials, m) chunk times and failed workers of the Sec. 4 simulations
    spawn key (8, count, N, m) random within-worker chunk orderings

Straggler patterns follow the simulation model of the paper's numerical
section: a worker processes its chunks in its fixed order, one chunk at a time,
with i.i.d. random per-chunk times; psi_j counts the chunks worker j has
finished by the deadline; failed workers have psi_j = 0.

Nothing here computes any part of the gradient-coding method (no coverage, no
coefficients, no gradients); the values returned are the stored inputs, in
their storage types, that both the GPU path and the oracle consume.
"""
from __future__ import annotations

import numpy as np
from scipy.special import gammaincinv

from .configs import Workload

PATTERN_BATCH = 1000


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=key)))


# ---------------------------------------------------------------------------
# regression data (workloads with n samples per chunk)
# ---------------------------------------------------------------------------

def chunk_X(wl: Workload, i: int, seed: int = 0) -> np.ndarray:
    """Chunk i of the design matrix, [n][d] fp32, entries N(0, x_std^2)."""
    z = _rng(seed, 0, i).standard_normal((wl.n, wl.d), dtype=np.float32)
    if wl.x_std != 1.0:
        z *= np.float32(wl.x_std)
    return z


def regression_data(wl: Workload, seed: int = 0, chunks=None):
    """X [N][n][d] fp32, y [N][n] fp32 and w [d] fp32 for a regression workload.

    Labels: linear y = X w* + N(0, noise_std^2); logistic y ~ Bernoulli(sigmoid(X w*)).
    ``chunks`` restricts generation to a subset of chunk indices (the labels of a
    chunk depend only on that chunk's rows, so subsets are consistent).
    """
    assert wl.n is not None and wl.loss in ("linear", "logistic")
    idx = list(range(wl.N)) if chunks is None else list(chunks)
    w_star = _rng(seed, 1).standard_normal(wl.d)
    noise_rng_states = _rng(seed, 2)
    # one noise draw of the full [N][n] shape keeps subsets consistent
    if wl.loss == "linear":
        noise = noise_rng_states.standard_normal((wl.N, wl.n)) * wl.noise_std
    else:
        noise = noise_rng_states.random((wl.N, wl.n))
    X = np.empty((len(idx), wl.n, wl.d), dtype=np.float32)
    y = np.empty((len(idx), wl.n), dtype=np.float32)
    for a, i in enumerate(idx):
        X[a] = chunk_X(wl, i, seed)
        z = X[a].astype(np.float64) @ w_star
        if wl.loss == "linear":
            y[a] = (z + noise[i]).astype(np.float32)
        else:
            p = 1.0 / (1.0 + np.exp(-z))
            y[a] = (noise[i] < p).astype(np.float32)
    if wl.w_std == 0.0:
        w = np.zeros(wl.d, dtype=np.float32)
    else:
        w = (_rng(seed, 3).standard_normal(wl.d) * wl.w_std).astype(np.float32)
    return X, y, w


def eval_points(wl: Workload, b: int, seed: int = 0) -> np.ndarray:
    """b evaluation points W [b][d] fp32 (row 0 is the workload's w)."""
    _, _, w0 = regression_data(wl, seed, chunks=[])
    W = np.empty((b, wl.d), dtype=np.float32)
    W[0] = w0
    if b > 1:
        std = wl.w_std if wl.w_std > 0 else 0.1
        W[1:] = (_rng(seed, 3, 1).standard_normal((b - 1, wl.d)) * std).astype(np.float32)
    return W


# ---------------------------------------------------------------------------
# chunk gradients given directly (bandwidth workloads)
# ---------------------------------------------------------------------------

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bfloat16 (round to nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def given_chunk(wl: Workload, i: int, seed: int = 0, cols=None) -> np.ndarray:
    """Chunk gradient i, i.i.d. N(0,1), in storage type (fp32, or bf16 bits as uint16).

    ``cols`` (a slice) returns only those entries, generating the row in full.
    """
    g = _rng(seed, 0, i).standard_normal(wl.d, dtype=np.float32)
    if cols is not None:
        g = g[cols]
    if wl.g_dtype == "bf16":
        return f32_to_bf16_bits(g)
    return g


def given_G(wl: Workload, seed: int = 0, chunks=None, threads: int = 1) -> np.ndarray:
    """Chunk gradients [len(chunks)][d] in storage type; chunks are independent streams,
    so ``threads`` > 1 generates them concurrently with identical values."""
    idx = list(range(wl.N)) if chunks is None else list(chunks)
    dt = np.uint16 if wl.g_dtype == "bf16" else np.float32
    G = np.empty((len(idx), wl.d), dtype=dt)

    def fill(a):
        G[a] = given_chunk(wl, idx[a], seed)

    if threads > 1:
        import concurrent.futures as cf
        with cf.ThreadPoolExecutor(threads) as ex:
            list(ex.map(fill, range(len(idx))))
    else:
        for a in range(len(idx)):
            fill(a)
    return G


# ---------------------------------------------------------------------------
# shared random matrix and straggler patterns
# ---------------------------------------------------------------------------

def shared_R(m: int, ell: int, seed: int = 0) -> np.ndarray:
    """R [ell][m] fp32 with i.i.d. N(0,1) entries (row k does not depend on ell)."""
    return _rng(seed, 4).standard_normal((ell, m)).astype(np.float32)


def _finished_by(cum_times: np.ndarray, deadline: np.ndarray) -> np.ndarray:
    """psi = number of chunks whose cumulative finish time is <= the deadline."""
    return np.sum(cum_times <= deadline[:, None, None], axis=2).astype(np.int32)


def _force_zero(rng: np.random.Generator, psi: np.ndarray, k: int) -> None:
    if k <= 0:
        return
    Pb, m = psi.shape
    order = np.argsort(rng.random((Pb, m)), axis=1)[:, :k]
    np.put_along_axis(psi, order, 0, axis=1)


def _median_deadline(cum_full: np.ndarray) -> np.ndarray:
    return np.median(cum_full, axis=1)


def worker_speeds(wl: Workload, seed: int = 0) -> np.ndarray:
    return _rng(seed, 5, 0).uniform(0.25, 1.0, size=wl.m)


def _pattern_batch(wl: Workload, b: int, Pb: int, variant: str, seed: int) -> np.ndarray:
    rng = _rng(seed, 5, 1 + b)
    m, delta = wl.m, wl.delta
    if wl.pattern == "uniform":
        # forced failures first, then uniform partial progress on {0..delta}
        forced = np.argsort(rng.random((Pb, m)), axis=1)[:, :wl.forced_zero] if wl.forced_zero else None
        psi = rng.integers(0, delta + 1, size=(Pb, m), dtype=np.int64).astype(np.int32)
        if forced is not None:
            np.put_along_axis(psi, forced, 0, axis=1)
        return psi
    if wl.pattern == "exp_median":
        tau = rng.exponential(1.0, size=(Pb, m, delta))
        cum = np.cumsum(tau, axis=2)
        return _finished_by(cum, _median_deadline(cum[:, :, -1]))
    if wl.pattern == "shifted_exp_fixed":
        tau = 1.0 + rng.exponential(1.0, size=(Pb, m, delta))
        cum = np.cumsum(tau, axis=2)
        T = delta + gammaincinv(delta, 0.5)
        return _finished_by(cum, np.full(Pb, T))
    if wl.pattern == "fail_exp_deadline":
        forced = np.argsort(rng.random((Pb, m)), axis=1)[:, :wl.forced_zero]
        tau = rng.exponential(1.0, size=(Pb, m, delta))
        psi = _finished_by(np.cumsum(tau, axis=2), np.full(Pb, wl.deadline))
        np.put_along_axis(psi, forced, 0, axis=1)
        return psi
    if wl.pattern == "hetero_median":
        speed = worker_speeds(wl, seed)
        tau = rng.exponential(1.0, size=(Pb, m, delta)) / speed[None, :, None]
        cum = np.cumsum(tau, axis=2)
        psi = _finished_by(cum, _median_deadline(cum[:, :, -1]))
        if variant == "ls":
            _force_zero(rng, psi, wl.ls_forced_zero)
        return psi
    raise ValueError(f"unknown pattern model {wl.pattern!r}")


def psi(wl: Workload, seed: int = 0, start: int = 0, count=None, variant: str = "exact") -> np.ndarray:
    """Straggler patterns [count][m] int32 for patterns start .. start+count-1.

    Patterns are generated in batches of PATTERN_BATCH with independent seeds,
    so any window of patterns is reproducible on its own.
    """
    if count is None:
        count = wl.P - start
    assert 0 <= start and start + count <= wl.P
    out = np.empty((count, wl.m), dtype=np.int32)
    p = start
    while p < start + count:
        b = p // PATTERN_BATCH
        b0 = b * PATTERN_BATCH
        Pb = min(PATTERN_BATCH, wl.P - b0)
        batch = _pattern_batch(wl, b, Pb, variant, seed)
        lo = p - b0
        hi = min(Pb, start + count - b0)
        out[p - start:p - start + hi - lo] = batch[lo:hi]
        p = b0 + hi
    return out


# ---------------------------------------------------------------------------
# random regular graphs (assignment supports of the regular-graph experiments)
# ---------------------------------------------------------------------------

def random_regular_graph(m: int, nu: int, seed: int = 0, attempt_limit: int = 1000) -> np.ndarray:
    """Adjacency matrix [m][m] (0/1, symmetric, zero diagonal) of a random nu-regular simple graph.

    Stubs are paired one random pair at a time among the pairs that create no loop
    and no repeated edge; a dead end restarts the pairing (the Steger-Wormald
    procedure).  Used as the assignment support A (chunk i on worker j iff edge ij),
    the kind of expander-based assignment of the paper's approximate-GC experiments.
    """
    if (m * nu) % 2 or nu >= m:
        raise ValueError("need m * nu even and nu < m")
    rng = _rng(seed, 6, m, nu)
    for _ in range(attempt_limit):
        A = np.zeros((m, m), dtype=np.int8)
        stubs = np.repeat(np.arange(m), nu)
        rng.shuffle(stubs)
        stubs = list(stubs)
        ok = True
        while stubs:
            placed = False
            for _try in range(50):
                a = int(rng.integers(len(stubs)))
                b = int(rng.integers(len(stubs)))
                u, v = stubs[a], stubs[b]
                if a != b and u != v and not A[u, v]:
                    A[u, v] = A[v, u] = 1
                    for k in sorted((a, b), reverse=True):
                        stubs[k] = stubs[-1]
                        stubs.pop()
                    placed = True
                    break
            if not placed:
                ok = False
                break
        if ok:
            return A
    raise RuntimeError("no simple regular graph found")


def random_orderings(A: np.ndarray, count: int, seed: int = 0) -> np.ndarray:
    """count ordering matrices [count][N][m] on the support A: every worker processes its
    chunks in an independent uniformly random order (positions 1..load of the worker)."""
    A = np.asarray(A) != 0
    N, m = A.shape
    rng = _rng(seed, 8, count, N, m)
    out = np.zeros((count, N, m), dtype=np.int32)
    for c in range(count):
        for j in range(m):
            rows = np.flatnonzero(A[:, j])
            out[c, rows, j] = rng.permutation(len(rows)) + 1
    return out


def chunk_times(wl: Workload, trials: int, seed: int = 0, failed: int | None = None):
    """The paper's simulation model, for time sweeps: per-chunk times tau [trials][m][delta]
    ~ i.i.d. Exp(1) (fp64) and a failure mask [trials][m] with `failed` workers chosen
    uniformly at random per trial (they never finish a chunk)."""
    rng = _rng(seed, 7, trials, wl.m)
    k = wl.forced_zero if failed is None else failed
    fail = np.zeros((trials, wl.m), dtype=bool)
    if k:
        idx = np.argsort(rng.random((trials, wl.m)), axis=1)[:, :k]
        np.put_along_axis(fail, idx, True, axis=1)
    tau = rng.exponential(1.0, size=(trials, wl.m, wl.delta))
    return tau, fail
