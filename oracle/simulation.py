"""Oracle: the straggler simulation of Sec. 4 (test infrastructure only).

Worker j processes the chunks of its order one after the other; the chunk at
position t (0-based) is finished at the cumulative time sum_{u <= t} tau_{j,u}
(Exp(1) chunk times in the paper's experiments); failed workers finish nothing.
At a deadline T the state vector psi(T) counts each worker's finished chunks.

Exact-GC completion time (the exact-GC simulation of Sec. 4): the first time T
at which every chunk has been processed at least ell times across the cluster.
The proposed protocol counts every processed chunk; original GC counts only
workers that have processed all their chunks.
"""
from __future__ import annotations

import numpy as np

from . import assignment


def progress(tau: np.ndarray, failed: np.ndarray | None, T: np.ndarray) -> np.ndarray:
    """psi [R][G][m]: chunks finished by each deadline T[g] (fp64 cumulative times)."""
    tau = np.asarray(tau, dtype=np.float64)
    cum = np.cumsum(tau, axis=2)                                  # [R][m][delta]
    psi = (cum[:, None, :, :] <= np.asarray(T, dtype=np.float64)[None, :, None, None]).sum(axis=3)
    if failed is not None:
        psi = np.where(np.asarray(failed, dtype=bool)[:, None, :], 0, psi)
    return psi.astype(np.int64)


def completion_time(tau_r: np.ndarray, failed_r: np.ndarray | None, O: np.ndarray, ell: int,
                    full_only: bool = False) -> float:
    """One trial, by an event sweep: process finish events in time order, count the copies
    of each chunk, and return the time at which the last chunk reaches ell copies
    (inf if it never does).  full_only: a worker's chunks all count at its completion time."""
    O = np.asarray(O)
    order, _, _ = assignment.tables(O)
    m, delta = order.shape
    cum = np.cumsum(np.asarray(tau_r, dtype=np.float64), axis=1)
    events = []
    for j in range(m):
        if failed_r is not None and failed_r[j]:
            continue
        for t in range(delta):
            i = order[j, t]
            if i < 0:
                continue
            when = cum[j, -1] if full_only else cum[j, t]
            events.append((when, i))
    events.sort()
    copies = np.zeros(O.shape[0], dtype=np.int64)
    short = O.shape[0]                     # chunks with fewer than ell copies
    for when, i in events:
        copies[i] += 1
        if copies[i] == ell:
            short -= 1
            if short == 0:
                return float(when)
    return float("inf")


def completion_times(tau: np.ndarray, failed: np.ndarray | None, O: np.ndarray, ell: int):
    """(partial [R], original [R]) completion times over trials."""
    R = tau.shape[0]
    f = [None] * R if failed is None else failed
    part = np.array([completion_time(tau[r], f[r], O, ell) for r in range(R)])
    orig = np.array([completion_time(tau[r], f[r], O, ell, full_only=True) for r in range(R)])
    return part, orig


def original_ls_error(O: np.ndarray, psi: np.ndarray) -> float:
    """Original GC's approximate decoding (the comparison of Sec. 4): with F the workers
    that have processed all their chunks, r = argmin ||A_F r - 1||_2 (r_j = 0 outside F),
    A the 0/1 assignment support; returns the squared residual ||A r - 1||^2."""
    O = np.asarray(O)
    psi = np.asarray(psi)
    A = (O != 0).astype(np.float64)
    loads = A.sum(axis=0)
    F = np.flatnonzero((psi >= loads) & (loads > 0))
    ones = np.ones(A.shape[0])
    if len(F) == 0:
        return float(A.shape[0])
    r = np.linalg.lstsq(A[:, F], ones, rcond=None)[0]
    res = A[:, F] @ r - ones
    return float(res @ res)
