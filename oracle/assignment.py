"""Oracle: assignment matrix support and chunk ordering (test infrastructure only).

Paper notation (Sec. 1 "Background"; Sec. 3 "Chunk Ordering Algorithm"):
    A  in R^{N x m}   A_ij != 0 iff chunk D_i is assigned to worker W_j
    O  in Z^{N x m}   O_ij = 0 if A_ij = 0, else the position (1..delta_j) of
                      D_i inside W_j, 1 = processed first
    gamma_i = nnz(A(i,:)) (replication),  delta_j = nnz(A(:,j)) (load)

Indices are 0-based here (chunk i, worker j); O keeps the paper's 1-based
positions so that O_ij = 0 still means "not assigned".

The tables used by the protocol are derived from O alone:
    order[j][t]   chunk at position t (0-based) of worker j, -1 past delta_j
    holder[i][u]  u-th worker holding chunk i (ascending worker index), -1 pad
    hpos[i][u]    0-based position of chunk i inside worker holder[i][u]
"""
from __future__ import annotations

import numpy as np


def cyclic_O(N: int, m: int, s: int) -> np.ndarray:
    """Ordering matrix of the cyclic scheme with N = m and load s + 1.

    Worker j holds chunks j, j+1, ..., j+s (mod N), processed in that order
    (the cyclic assignment of the original gradient-coding scheme, whose
    ordering Sec. 3 states is optimal for exact GC).  So O[(j+t) mod N, j] = t+1.
    """
    if N != m:
        raise ValueError("the cyclic scheme has N = m")
    if not 0 <= s < m:
        raise ValueError("need 0 <= s < m")
    O = np.zeros((N, m), dtype=np.int64)
    for j in range(m):
        for t in range(s + 1):
            O[(j + t) % N, j] = t + 1
    return O


def check_O(O: np.ndarray) -> None:
    """An ordering matrix: in every column the non-zero values are 1..delta_j, once each."""
    O = np.asarray(O)
    if O.ndim != 2 or (O < 0).any():
        raise ValueError("O must be a non-negative 2-D integer matrix")
    for j in range(O.shape[1]):
        vals = sorted(int(v) for v in O[:, j] if v != 0)
        if vals != list(range(1, len(vals) + 1)):
            raise ValueError(f"column {j} of O is not an ordering")


def loads(O: np.ndarray) -> np.ndarray:
    """delta_j = nnz(A(:, j))."""
    return (np.asarray(O) != 0).sum(axis=0)


def replications(O: np.ndarray) -> np.ndarray:
    """gamma_i = nnz(A(i, :))."""
    return (np.asarray(O) != 0).sum(axis=1)


def tables(O: np.ndarray, delta: int | None = None, gamma: int | None = None):
    """order [m][delta], holder [N][gamma], hpos [N][gamma] (int32, -1 padded)."""
    O = np.asarray(O)
    check_O(O)
    N, m = O.shape
    delta = int(loads(O).max()) if delta is None else delta
    gamma = int(replications(O).max()) if gamma is None else gamma
    order = np.full((m, delta), -1, dtype=np.int32)
    holder = np.full((N, gamma), -1, dtype=np.int32)
    hpos = np.full((N, gamma), -1, dtype=np.int32)
    for j in range(m):
        for i in range(N):
            if O[i, j]:
                order[j, O[i, j] - 1] = i
    for i in range(N):
        u = 0
        for j in range(m):
            if O[i, j]:
                holder[i, u] = j
                hpos[i, u] = O[i, j] - 1
                u += 1
    return order, holder, hpos


def Q(O: np.ndarray) -> np.ndarray:
    """Q_i(O): the most chunks the cluster can process with no copy of D_i processed (Sec. 3).

    Worker j can process everything above D_i's position (O_ij - 1 chunks) when
    it holds D_i, and all of its delta chunks otherwise.  For a delta-regular
    assignment this is the paper's closed form; here it is counted directly.
    """
    O = np.asarray(O)
    d = loads(O)
    out = np.zeros(O.shape[0], dtype=np.int64)
    for i in range(O.shape[0]):
        out[i] = sum(int(O[i, j]) - 1 if O[i, j] else int(d[j]) for j in range(O.shape[1]))
    return out
