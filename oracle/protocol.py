"""Oracle: the partial-straggler gradient-coding protocol (test infrastructure only).

Written from Sec. 2 ("Gradient Coding for partial stragglers"), Sec. 2.1
("Analysis of Algorithm 1") and Sec. 2.2 ("Illustrative Example") of the paper.
All arithmetic is fp64; inputs are the stored fp32 (or bf16) values widened.
Indices are 0-based; the paper's W_1..W_m, D_1..D_N are workers 0..m-1 and
chunks 0..N-1 here.

Notation:
    psi [m]        chunks processed by each worker when the PS broadcasts the
                   encode-and-transmit signal; W_j has processed the chunks at
                   positions 1..psi_j of its order
    S_i            workers that processed D_i;  Delta_i = |S_i|
    R [ell][m]     the shared N(0,1) matrix
    B [m][N*ell]   the matrix of indeterminates (block column B^(i) holds the
                   ell columns that weight the blocks g_{D_i}[0..ell-1])
    g[k]           block k of a gradient: entries [k*L, (k+1)*L) of the
                   gradient zero-padded to length ell*L, L = ceil(d / ell)
    T [m][L]       g_beta, the vector worker beta transmits
"""
from __future__ import annotations

import numpy as np

from . import assignment


# ---------------------------------------------------------------------------
# inputs
# ---------------------------------------------------------------------------

def widen(G: np.ndarray, dtype: str = "f32") -> np.ndarray:
    """Stored chunk gradients -> fp64.  bf16 values are given as their uint16 bit patterns."""
    if dtype == "bf16":
        bits = np.asarray(G, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    return np.asarray(G, dtype=np.float64)


def check_psi(O: np.ndarray, psi: np.ndarray) -> bool:
    """psi is a valid state vector: 0 <= psi_j <= delta_j for every worker."""
    psi = np.asarray(psi)
    return bool(((psi >= 0) & (psi <= assignment.loads(O))).all())


# ---------------------------------------------------------------------------
# global state shared through psi (Sec. 2, protocol description)
# ---------------------------------------------------------------------------

def processed(O: np.ndarray, psi: np.ndarray) -> np.ndarray:
    """[N][m] bool: W_j has processed D_i, i.e. D_i sits at a position <= psi_j of W_j."""
    O = np.asarray(O)
    psi = np.asarray(psi)
    if not check_psi(O, psi):
        raise ValueError("psi out of range")
    return (O != 0) & (O <= psi[None, :])


def processed_sets(O: np.ndarray, psi: np.ndarray):
    """S_i for every chunk, as ascending worker indices (Sec. 2.1, exact GC analysis)."""
    Pm = processed(O, psi)
    return [np.flatnonzero(Pm[i]) for i in range(Pm.shape[0])]


def coverage(O: np.ndarray, psi: np.ndarray) -> np.ndarray:
    """Delta_i: the number of processed copies of D_i across the cluster."""
    return processed(O, psi).sum(axis=1).astype(np.int64)


def decodable(O: np.ndarray, psi: np.ndarray, ell: int) -> bool:
    """Exact recovery is possible when every chunk has been processed at least ell times.

    This is the condition under which the PS sends the encode-and-transmit
    signal for exact GC (Sec. 2); Sec. 2.1 shows each ell x Delta_i system is
    then solvable.  Decided in integers.
    """
    return bool((coverage(O, psi) >= ell).all())


def coef_err(O: np.ndarray, psi: np.ndarray, ell: int) -> int:
    """sum_i max(0, ell - Delta_i): the total coefficient-space error (end of Sec. 2.1)."""
    return int(np.maximum(0, ell - coverage(O, psi)).sum())


def indeterminate_support(O: np.ndarray, psi: np.ndarray, ell: int) -> np.ndarray:
    """[m][N*ell] bool: row j of block column B^(i) holds indeterminates iff W_j processed D_i."""
    Pm = processed(O, psi)          # [N][m]
    return np.repeat(Pm.T, ell, axis=1)


# ---------------------------------------------------------------------------
# Algorithm 1 (Find-Encoding-Coeff)
# ---------------------------------------------------------------------------

def worker_solve(beta: int, O: np.ndarray, psi: np.ndarray, R: np.ndarray) -> dict:
    """Algorithm 1 as run by worker W_beta.

    Steps: form the indeterminate support of B from psi; keep the block
    columns of the chunks W_beta has processed (B~_beta, eq. of the extracted
    block columns); choose the indeterminates of B~_beta as the minimum-l2-norm
    least-squares solution of  min || 1^T (x) I_ell - R B~_beta ||  (the norm of
    a matrix read as the Frobenius norm).  Returns {(i, j, k): value} for every
    indeterminate of B~_beta: chunk i, worker j, column k of B^(i).
    """
    R = np.asarray(R, dtype=np.float64)
    ell = R.shape[0]
    Pm = processed(O, psi)
    chunks = [i for i in range(Pm.shape[0]) if Pm[i, beta]]          # ascending, as in B~_beta
    unknowns = [(i, j, k) for i in chunks for j in np.flatnonzero(Pm[i]) for k in range(ell)]
    if not unknowns:
        return {}
    col = {u: c for c, u in enumerate(unknowns)}
    # residual entries: (R B~)[r, (i, k)] - [r == k]
    rows = [(i, k, r) for i in chunks for k in range(ell) for r in range(ell)]
    A = np.zeros((len(rows), len(unknowns)))
    b = np.zeros(len(rows))
    for a, (i, k, r) in enumerate(rows):
        b[a] = 1.0 if r == k else 0.0
        for j in np.flatnonzero(Pm[i]):
            A[a, col[(i, j, k)]] = R[r, j]
    x = np.linalg.lstsq(A, b, rcond=None)[0]
    return {u: x[c] for u, c in col.items()}


def encoding_matrix(O: np.ndarray, psi: np.ndarray, R: np.ndarray) -> np.ndarray:
    """B [m][N*ell]: row beta is epsilon_beta, the row W_beta keeps from its own solve."""
    O = np.asarray(O)
    R = np.asarray(R, dtype=np.float64)
    ell = R.shape[0]
    N, m = O.shape
    B = np.zeros((m, N * ell))
    for beta in range(m):
        for (i, j, k), v in worker_solve(beta, O, psi, R).items():
            if j == beta:
                B[beta, i * ell + k] = v
    return B


def encoding_matrix_per_chunk(O: np.ndarray, psi: np.ndarray, R: np.ndarray) -> np.ndarray:
    """B assembled chunk by chunk: B^(i) restricted to S_i is the pseudo-inverse of R[:, S_i].

    The Frobenius objective of Algorithm 1 separates into one least-squares
    problem per column of every B^(i) (Sec. 2.1 and the W_5 example of
    Sec. 2.2); their minimum-norm solutions stacked are pinv(R[:, S_i]).  Used
    only as a second route to cross-check ``encoding_matrix``.
    """
    O = np.asarray(O)
    R = np.asarray(R, dtype=np.float64)
    ell = R.shape[0]
    N, m = O.shape
    B = np.zeros((m, N * ell))
    for i, S in enumerate(processed_sets(O, psi)):
        if len(S):
            B[S, i * ell:(i + 1) * ell] = np.linalg.pinv(R[:, S])
    return B


def compact(B: np.ndarray, O: np.ndarray, ell: int) -> np.ndarray:
    """Bc [m][delta][ell]: Bc[j][t][k] = B^(order[j][t])_{j,k}, the weight W_j gives block k
    of its t-th chunk (zero past delta_j; zero for unprocessed positions since B is)."""
    order, _, _ = assignment.tables(O)
    m, delta = order.shape
    Bc = np.zeros((m, delta, ell))
    for j in range(m):
        for t in range(delta):
            i = order[j, t]
            if i >= 0:
                Bc[j, t, :] = B[j, i * ell:(i + 1) * ell]
    return Bc


def coef_residual(B: np.ndarray, R: np.ndarray) -> float:
    """|| 1_N^T (x) I_ell - R B ||_F^2, the coefficient-space error of a coding matrix B."""
    R = np.asarray(R, dtype=np.float64)
    ell, m = R.shape
    N = B.shape[1] // ell
    target = np.tile(np.eye(ell), (1, N))
    return float(np.sum((target - R @ B) ** 2))


# ---------------------------------------------------------------------------
# encode (workers) and combine (PS)
# ---------------------------------------------------------------------------

def blocks(g: np.ndarray, ell: int) -> np.ndarray:
    """g[0..ell-1] as an [ell][L] array: contiguous blocks of the zero-padded vector."""
    g = np.asarray(g, dtype=np.float64)
    d = g.shape[-1]
    L = -(-d // ell)
    pad = np.zeros(g.shape[:-1] + (ell * L,))
    pad[..., :d] = g
    return pad.reshape(g.shape[:-1] + (ell, L))


def encode(B: np.ndarray, G: np.ndarray, ell: int) -> np.ndarray:
    """T[beta] = g_beta = sum_i sum_k B^(i)_{beta,k} g_{D_i}[k]  (Sec. 2, worker encode)."""
    Gb = blocks(G, ell)                       # [N][ell][L]
    N, _, L = Gb.shape
    return B @ Gb.reshape(N * ell, L)


def reconstruct(T: np.ndarray, R: np.ndarray, d: int) -> np.ndarray:
    """PS combine: block k of the estimate is sum_j R[k, j] g_j  (Sec. 2.2, last step)."""
    R = np.asarray(R, dtype=np.float64)
    return (R @ T).reshape(-1)[:d]


def reconstruct_by_chunks(B: np.ndarray, R: np.ndarray, G: np.ndarray) -> np.ndarray:
    """Second route: sum_i of block-mixed chunk gradients, (R B^(i)) applied to g_{D_i}'s blocks.

    Equal to ``reconstruct(encode(B, G))`` by associativity; a cross-check only.
    """
    R = np.asarray(R, dtype=np.float64)
    ell = R.shape[0]
    Gb = blocks(G, ell)
    N, _, L = Gb.shape
    d = np.asarray(G).shape[-1]
    acc = np.zeros((ell, L))
    for i in range(N):
        acc += (R @ B[:, i * ell:(i + 1) * ell]) @ Gb[i]
    return acc.reshape(-1)[:d]


# ---------------------------------------------------------------------------
# one straggler pattern end to end
# ---------------------------------------------------------------------------

def run_pattern(O: np.ndarray, psi: np.ndarray, R: np.ndarray, G: np.ndarray | None = None) -> dict:
    """Coverage, decodability, coefficients and (given G [N][d] fp64) T, the estimate and its error."""
    R = np.asarray(R, dtype=np.float64)
    ell = R.shape[0]
    out = {
        "cov": coverage(O, psi),
        "dec": decodable(O, psi, ell),
        "coef_err": coef_err(O, psi, ell),
    }
    B = encoding_matrix(O, psi, R)
    out["B"] = B
    out["Bc"] = compact(B, O, ell)
    if G is not None:
        G = np.asarray(G, dtype=np.float64)
        T = encode(B, G, ell)
        ghat = reconstruct(T, R, G.shape[1])
        out["T"] = T
        out["ghat"] = ghat
        out["sqerr"] = float(np.sum((ghat - G.sum(axis=0)) ** 2))
    return out
