"""Batched drivers around the oracle for the parity tests (test infrastructure).

Loops the per-pattern oracle functions over many patterns and computes the
forward-error bounds the GPU results are held to.  Uses only ``oracle`` and
``workloads``.
"""
from __future__ import annotations

import numpy as np

import oracle.assignment as OA
import oracle.gradients as OG
import oracle.protocol as OP

U = 2.0 ** -24          # unit roundoff of fp32 (round to nearest)


def gamma(n):
    """gamma_n = n u / (1 - n u): the classical bound factor for n fp32 roundings."""
    n = np.asarray(n, dtype=np.float64)
    return n * U / (1.0 - n * U)


def encode_bound(nterm, M, g_dtype="f32"):
    """Elementwise bound on the GPU encode's |T - T_ref| for rows with nterm = psi*ell terms
    of magnitude sum M = sum_{t,k} |Bc||g|.  Every path may run on the bf16 matrix cores,
    where each fp32 coefficient a is split by rounding into three bf16 parts (leaving at most
    u|a|), the parts' products are exact in fp32 and are accumulated in fp32, each
    accumulation allowed 2u (the matrix cores' rounding of their internal sums is not assumed
    to be to nearest): gamma'_k = 2ku / (1 - 2ku).
    bf16 chunk gradients: three products per term, u M + gamma'_{3n+1} M.
    fp32 chunk gradients: each g is split exactly into three bf16 parts by truncation
    (|g2| < 2^-7 |g|, |g3| < 2^-14 |g|) and six of the nine products are kept; the three
    dropped ones and the coefficient's residue stay below 8u |a||g| per term, and the kept
    ones sum to at most 1.02 |a||g|: 8u M + 1.02 gamma'_{6n+1} M.  Both also bound the
    vector path's gamma_n M."""
    return encode_eps(nterm, g_dtype)[..., None] * M


def encode_eps(nterm, g_dtype="f32"):
    """The factor of encode_bound: u + gamma'_{3n+1} (bf16), 8u + 1.02 gamma'_{6n+1} (fp32)."""
    nterm = np.asarray(nterm, dtype=np.float64)
    if g_dtype == "bf16":
        k = 3 * nterm + 1
        return U + 2 * k * U / (1.0 - 2 * k * U)
    k = 6 * nterm + 1
    return 8 * U + 1.02 * 2 * k * U / (1.0 - 2 * k * U)


def coverage_all(O, psi):
    """cov [P][N], dec [P] (for each ell given later), via the oracle per pattern."""
    return np.stack([OP.coverage(O, p) for p in psi]).astype(np.int64)


def coefficients(O, psi, R, per_worker=False):
    """Bc [P][m][delta][ell] fp64 and the per-(pattern, chunk) 2-norm condition numbers
    of R[:, S_i] (0 where Delta_i = 0)."""
    R = np.asarray(R, dtype=np.float64)
    ell = R.shape[0]
    N, m = O.shape
    Bcs, kappas = [], []
    for p in psi:
        B = OP.encoding_matrix(O, p, R) if per_worker else OP.encoding_matrix_per_chunk(O, p, R)
        Bcs.append(OP.compact(B, O, ell))
        kap = np.zeros(N)
        for i, S in enumerate(OP.processed_sets(O, p)):
            if len(S):
                kap[i] = np.linalg.cond(R[:, S])
        kappas.append(kap)
    return np.stack(Bcs), np.stack(kappas)


def bc_bound(Bc_ref, kappa, O):
    """Elementwise bound for the GPU's Bc: one fp32 rounding of the fp64 value plus the
    fp64 Gram/Cholesky solve's error, which grows like kappa^2 * 2^-53 times the block's size."""
    order, _, _ = OA.tables(O)
    P, m, delta, ell = Bc_ref.shape
    out = 2 * U * np.abs(Bc_ref)
    for p in range(P):
        for j in range(m):
            for t in range(delta):
                i = order[j, t]
                if i < 0:
                    continue
                out[p, j, t, :] += 1e-14 * max(1.0, kappa[p, i]) ** 2 * (np.abs(Bc_ref[p, j, t, :]).max() + 1e-300)
    return out


def gblocks(G, ell):
    return OP.blocks(np.asarray(G, dtype=np.float64), ell)       # [N][ell][L]


def encode_ref(Bc, psi, order, G, ell):
    """T [P][m][L] from compact coefficients over each worker's processed prefix (fp64),
    and its magnitude sum_{t,k} |Bc||g| for the error bound."""
    Gb = gblocks(G, ell)
    N, _, L = Gb.shape
    P, m, delta, _ = Bc.shape
    T = np.zeros((P, m, L))
    M = np.zeros((P, m, L))
    n_terms = np.zeros((P, m))
    for p in range(P):
        for j in range(m):
            npj = min(max(int(psi[p, j]), 0), delta)
            for t in range(npj):
                c = order[j, t]
                if c < 0:
                    continue
                for k in range(ell):
                    T[p, j] += Bc[p, j, t, k] * Gb[c, k]
                    M[p, j] += abs(Bc[p, j, t, k]) * np.abs(Gb[c, k])
                    n_terms[p, j] += 1
    return T, M, n_terms


def reconstruct_ref(T, R, d):
    R = np.asarray(R, dtype=np.float64)
    P, m, L = T.shape
    gh = np.einsum("km,pml->pkl", R, T).reshape(P, -1)[:, :d]
    mag = np.einsum("km,pml->pkl", np.abs(R), np.abs(T)).reshape(P, -1)[:, :d]
    return gh, mag


def end_to_end(O, psi, R, G, per_worker=False):
    """Full oracle: coefficients from psi and R, encode, combine.  Returns ghat [P][d]."""
    R = np.asarray(R, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    out = []
    for p in psi:
        B = OP.encoding_matrix(O, p, R) if per_worker else OP.encoding_matrix_per_chunk(O, p, R)
        out.append(OP.reconstruct(OP.encode(B, G, R.shape[0]), R, G.shape[1]))
    return np.stack(out)


def chunk_grads(X, y, W, loss):
    return OG.chunk_gradients(X, y, W, loss)


def sampled_blocks(G, dtype, ell, xs):
    """Columns of the chunk gradients that block positions xs (in [0, L)) touch, laid out so
    that ``OP.blocks(Gsub, ell)`` has block k = entries k*L + xs of the zero-padded gradients.
    Lets the oracle compute T[:, xs] and the estimate at k*L + xs one by one at any d."""
    G = np.asarray(G)
    N, d = G.shape
    L = -(-d // ell)
    S = len(xs)
    Gsub = np.zeros((N, ell * S))
    for k in range(ell):
        for s_, x in enumerate(xs):
            c = k * L + int(x)
            if c < d:
                Gsub[:, k * S + s_] = OP.widen(G[:, c], dtype)
    return Gsub


def mixing(O, psi, R):
    """M [N][ell][ell] fp64 with M_i = R B^(i): how chunk i's blocks enter the estimate, from the
    oracle's coefficients (``reconstruct_by_chunks`` sums M_i applied to g_i's blocks)."""
    R = np.asarray(R, dtype=np.float64)
    ell = R.shape[0]
    B = OP.encoding_matrix_per_chunk(O, psi, R)
    N = O.shape[0]
    return np.stack([R @ B[:, i * ell:(i + 1) * ell] for i in range(N)])


def direct_ref(O, psi, R, G):
    """The estimate sum_i M_i g_i (fp64) of each pattern, with sum_i |M_i| |g_i| for its error
    bound and the largest condition number of an R[:, S_i] with 0 < Delta_i < ell."""
    R = np.asarray(R, dtype=np.float64)
    ell = R.shape[0]
    G = np.asarray(G, dtype=np.float64)
    d = G.shape[1]
    Gb = gblocks(G, ell)                                             # [N][ell][L]
    out, mag, kap = [], [], []
    for p in psi:
        M = mixing(O, p, R)
        out.append(np.einsum("ikq,iql->kl", M, Gb).reshape(-1)[:d])
        mag.append(np.einsum("ikq,iql->kl", np.abs(M), np.abs(Gb)).reshape(-1)[:d])
        c = OP.coverage(O, p)
        k = [np.linalg.cond(R[:, S]) for S, n in zip(OP.processed_sets(O, p), c) if 0 < n < ell]
        kap.append(max(k + [1.0]))
    return np.stack(out), np.stack(mag), np.array(kap)
