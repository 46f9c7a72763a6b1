"""Planted mistakes in the oracle (on the CPU) must each be caught by at least one pin.

Every mutant replaces one oracle function with a plausible slip (an off-by-one,
a dropped term, a wrong sign, index or operand) and runs the pins; the test
passes when some pin fails.  This shows the pins constrain every step.
"""
import numpy as np
import pytest

import oracle.assignment as OA
import oracle.gradients as OG
import oracle.ordering as OO
import oracle.protocol as OP
import oracle.simulation as OS
import pins

_orig_processed = OP.processed
_orig_worker_solve = OP.worker_solve
_orig_encode = OP.encode
_orig_cyclic = OA.cyclic_O
_orig_compact = OP.compact


def m_processed_offbyone(O, psi):
    return (np.asarray(O) != 0) & (np.asarray(O) < np.asarray(psi)[None, :])


def m_coverage_ignores_psi(O, psi):
    return (np.asarray(O) != 0).sum(axis=1)


def m_coef_err_sign(O, psi, ell):
    return int(np.maximum(0, OP.coverage(O, psi) - ell).sum())


def m_decodable_strict(O, psi, ell):
    return bool((OP.coverage(O, psi) > ell).all())


def m_worker_solve_target(beta, O, psi, R):
    # drops the off-diagonal rows of the target: solves only for r == k
    sol = _orig_worker_solve(beta, O, psi, R[:1])
    ell = np.asarray(R).shape[0]
    return {(i, j, k): v for (i, j, _), v in sol.items() for k in range(ell)}


def m_encode_drop_last_chunk(B, G, ell):
    B = B.copy()
    B[:, -ell:] = 0.0
    return _orig_encode(B, G, ell)


def m_reconstruct_rows_swapped(T, R, d):
    R = np.asarray(R, dtype=np.float64)[::-1]
    return (R @ T).reshape(-1)[:d]


def m_reconstruct_transposed_blocks(T, R, d):
    R = np.asarray(R, dtype=np.float64)
    return (R @ T).T.reshape(-1)[:d]


def m_blocks_strided(g, ell):
    g = np.asarray(g, dtype=np.float64)
    d = g.shape[-1]
    L = -(-d // ell)
    pad = np.zeros(g.shape[:-1] + (ell * L,))
    pad[..., :d] = g
    return np.swapaxes(pad.reshape(g.shape[:-1] + (L, ell)), -1, -2)


def m_cyclic_reversed(N, m, s):
    O = _orig_cyclic(N, m, s)
    return np.where(O > 0, s + 2 - O, 0)


def m_compact_shifted(B, O, ell):
    Bc = _orig_compact(B, O, ell)
    return np.roll(Bc, 1, axis=1)


def m_widen_low_half(G, dtype="f32"):
    if dtype == "bf16":
        bits = np.asarray(G, dtype=np.uint16).astype(np.uint32)
        return bits.view(np.float32).astype(np.float64)
    return np.asarray(G, dtype=np.float64)


_orig_ordering = OO.chunk_ordering


def m_ordering_unweighted(A):
    O = _orig_ordering(A)
    return (O != 0).astype(np.int64)           # drops the weights i of O = sum_i i P_i


def m_ordering_greedy(A):
    # takes, for every chunk in turn, the first worker still free: not a matching step
    S = np.asarray(A) != 0
    N, m = S.shape
    delta = int(S.sum(axis=0)[0])
    O = np.zeros((N, m), dtype=np.int64)
    for j in range(m):
        rows = np.flatnonzero(S[:, j])
        for t, i in enumerate(rows):
            O[i, j] = t + 1
    return O


_orig_completion = OS.completion_time


def m_completion_off_by_one(tau_r, failed_r, O, ell, full_only=False):
    # stops at ell - 1 copies
    return _orig_completion(tau_r, failed_r, O, max(1, ell - 1), full_only) if ell > 1 else \
        _orig_completion(tau_r, failed_r, O, ell, not full_only)


def m_progress_strict(tau, failed, T):
    tau = np.asarray(tau, dtype=np.float64)
    cum = np.cumsum(tau, axis=2)
    psi = (cum[:, None, :, :] < np.asarray(T)[None, :, None, None]).sum(axis=3)
    if failed is not None:
        psi = np.where(np.asarray(failed, dtype=bool)[:, None, :], 0, psi)
    return psi


def m_grad_sign(Xi, yi, w, loss):
    Xi = np.asarray(Xi, dtype=np.float64)
    z = Xi @ np.asarray(w, dtype=np.float64)
    r = (np.asarray(yi) - z) if loss == "linear" else (np.asarray(yi) - OG.sigmoid(z))
    return Xi.T @ r


def m_grad_no_sigmoid(Xi, yi, w, loss):
    Xi = np.asarray(Xi, dtype=np.float64)
    z = Xi @ np.asarray(w, dtype=np.float64)
    return Xi.T @ (z - np.asarray(yi))


def m_grad_residual_misindexed(Xi, yi, w, loss):
    # pairs sample r's features with sample (n-1-r)'s residual: an index slip
    Xi = np.asarray(Xi, dtype=np.float64)
    z = Xi @ np.asarray(w, dtype=np.float64)
    r = z - yi if loss == "linear" else OG.sigmoid(z) - yi
    return Xi.T @ r[::-1]


MUTANTS = [
    (OP, "processed", m_processed_offbyone),
    (OP, "coverage", m_coverage_ignores_psi),
    (OP, "coef_err", m_coef_err_sign),
    (OP, "decodable", m_decodable_strict),
    (OP, "worker_solve", m_worker_solve_target),
    (OP, "encode", m_encode_drop_last_chunk),
    (OP, "reconstruct", m_reconstruct_rows_swapped),
    (OP, "reconstruct", m_reconstruct_transposed_blocks),
    (OP, "blocks", m_blocks_strided),
    (OA, "cyclic_O", m_cyclic_reversed),
    (OP, "compact", m_compact_shifted),
    (OP, "widen", m_widen_low_half),
    (OO, "chunk_ordering", m_ordering_unweighted),
    (OO, "chunk_ordering", m_ordering_greedy),
    (OS, "completion_time", m_completion_off_by_one),
    (OS, "progress", m_progress_strict),
    (OG, "chunk_gradient", m_grad_sign),
    (OG, "chunk_gradient", m_grad_no_sigmoid),
    (OG, "chunk_gradient", m_grad_residual_misindexed),
]


def _some_pin_fails():
    for pin in pins.ALL_PINS + [lambda: pins.pin_bruteforce_decodability(cases=[(3, 1), (4, 1)])]:
        try:
            pin()
        except (AssertionError, ValueError, IndexError, KeyError):
            return True
    return False


@pytest.mark.parametrize("mod,name,mutant", MUTANTS, ids=[f"{n}:{f.__name__}" for _, n, f in MUTANTS])
def test_mutant_is_caught(monkeypatch, mod, name, mutant):
    monkeypatch.setattr(mod, name, mutant)
    assert _some_pin_fails(), f"no pin caught the planted mistake {mutant.__name__}"


def test_unmutated_oracle_passes_every_pin():
    assert not _some_pin_fails()
