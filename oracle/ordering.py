"""Oracle: Algorithm 2 (Chunk-Ordering) of Sec. 3 (test infrastructure only).

For an assignment with N = m and every chunk and worker of degree delta (a
delta-regular bipartite graph between chunks and workers), Algorithm 2 peels
delta perfect matchings P_1, ..., P_delta off the support (Claim 1: a
delta-regular bipartite graph always has one, by Hall's condition) and sets
O = sum_i i * P_i.  Every row of O then sums to delta(delta+1)/2, the lower
bound on max_i sum_j O_ij shown in Sec. 3, so Q_max is optimal.

Matchings here are found with plain augmenting paths (Kuhn's method); any
perfect matching is a valid step, so orderings are not unique -- only their
validity and their Q_max are.
"""
from __future__ import annotations

import numpy as np


def perfect_matching(S: np.ndarray) -> np.ndarray:
    """A perfect matching of the bipartite graph with biadjacency S (rows = chunks,
    columns = workers), as match[i] = worker matched to chunk i.  Raises if none exists."""
    S = np.asarray(S, dtype=bool)
    N, m = S.shape
    owner = [-1] * m                       # worker -> chunk

    def augment(i, seen):
        for j in np.flatnonzero(S[i]):
            if not seen[j]:
                seen[j] = True
                if owner[j] < 0 or augment(owner[j], seen):
                    owner[j] = i
                    return True
        return False

    for i in range(N):
        if not augment(i, [False] * m):
            raise ValueError("no perfect matching")
    match = np.full(N, -1, dtype=np.int64)
    for j, i in enumerate(owner):
        if i >= 0:
            match[i] = j
    return match


def chunk_ordering(A: np.ndarray) -> np.ndarray:
    """Algorithm 2: the ordering matrix O for a delta-regular support A (N = m)."""
    S = np.asarray(A) != 0
    N, m = S.shape
    if N != m:
        raise ValueError("Algorithm 2 needs N = m")
    deg = S.sum(axis=0)
    delta = int(deg[0]) if m else 0
    if not ((S.sum(axis=1) == delta).all() and (deg == delta).all()):
        raise ValueError("support is not delta-regular")
    O = np.zeros((N, m), dtype=np.int64)
    cur = S.copy()
    for step in range(1, delta + 1):
        match = perfect_matching(cur)          # P_step
        for i in range(N):
            O[i, match[i]] = step
            cur[i, match[i]] = False
    return O


def q_max(O: np.ndarray) -> int:
    """Q_max(O) = max_i Q_i(O), Q_i counted directly (Sec. 3)."""
    from .assignment import Q
    return int(Q(O).max())
