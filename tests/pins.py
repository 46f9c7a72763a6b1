"""Pins that tie the oracle to what the paper and the mathematics fix.

Each ``pin_*`` function raises AssertionError when the oracle disagrees with a
worked example of the paper, a closed form, an invariant, a special case that
reduces to a textbook result, or a brute-force enumeration.  The functions
reach the oracle through its module attributes at call time, so the mutation
tests can plant a mistake in the oracle and check that some pin catches it.
"""
from __future__ import annotations

import itertools
import math
import os

import numpy as np

import oracle.assignment as OA
import oracle.gradients as OG
import oracle.ordering as OO
import oracle.protocol as OP
import oracle.simulation as OS

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_rows(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([int(v) for v in line.split()])
    return rows


def sec2_2_O():
    """Ordering matrix of the Sec. 2.2 example from the orders read in sec2_2_orders.txt."""
    orders = load_rows("sec2_2_orders.txt")
    O = np.zeros((5, 5), dtype=np.int64)
    for j, chunks in enumerate(orders):
        for t, c in enumerate(chunks):
            O[c - 1, j] = t + 1
    return O


def rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------------------
# assignment
# ---------------------------------------------------------------------------

def pin_fig1a_ordering():
    O = OA.cyclic_O(3, 3, 1)
    assert (O == np.array(load_rows("fig1a_cyclic_m3_s1.txt"))).all()


CYCLIC_CASES = [(3, 1), (4, 1), (5, 2), (6, 2), (20, 3), (50, 4), (100, 9), (200, 19), (7, 0), (9, 8)]


def pin_cyclic_invariants():
    for m, s in CYCLIC_CASES:
        delta = s + 1
        O = OA.cyclic_O(m, m, s)
        # every worker holds delta distinct chunks at positions 1..delta, every chunk gamma = s+1 copies
        for j in range(m):
            assert sorted(O[:, j][O[:, j] > 0].tolist()) == list(range(1, delta + 1))
        assert ((O > 0).sum(axis=1) == delta).all()
        # Sec. 3: every row sum attains the lower bound delta(delta+1)/2 on Q_max's variable part
        assert (O.sum(axis=1) == delta * (delta + 1) // 2).all()
        # Sec. 3 closed form of Q_i for a delta-regular assignment
        assert (OA.Q(O) == O.sum(axis=1) + (m - delta - 1) * delta).all()
        order, holder, hpos = OA.tables(O)
        for j in range(m):
            for t in range(delta):
                assert order[j, t] == (j + t) % m          # W_j processes j, j+1, ..., j+s in order
        for i in range(m):
            assert sorted(holder[i].tolist()) == sorted(((i - t) % m) for t in range(delta))
            for u in range(delta):
                assert order[holder[i, u], hpos[i, u]] == i


def pin_tables_roundtrip():
    g = rng(1)
    for _ in range(20):
        N, m = g.integers(2, 9, size=2)
        A = g.random((N, m)) < 0.5
        O = np.zeros((N, m), dtype=np.int64)
        for j in range(m):
            rows = np.flatnonzero(A[:, j])
            g.shuffle(rows)
            for t, i in enumerate(rows):
                O[i, j] = t + 1
        order, holder, hpos = OA.tables(O)
        back = np.zeros_like(O)
        for j in range(m):
            for t in range(order.shape[1]):
                if order[j, t] >= 0:
                    back[order[j, t], j] = t + 1
        assert (back == O).all()
        for i in range(N):
            for u in range(holder.shape[1]):
                if holder[i, u] >= 0:
                    assert O[i, holder[i, u]] == hpos[i, u] + 1


# ---------------------------------------------------------------------------
# chunk gradients
# ---------------------------------------------------------------------------

def _tiny_regression(seed, N=3, n=5, d=7, logistic=False):
    g = rng(seed)
    X = g.standard_normal((N, n, d))
    if logistic:
        y = (g.random((N, n)) < 0.5).astype(np.float64)
    else:
        y = g.standard_normal((N, n))
    return X, y


def _sample_loss(x, y, w, loss):
    z = sum(a * b for a, b in zip(x, w))
    if loss == "linear":
        return 0.5 * (z - y) ** 2
    # Bernoulli negative log-likelihood of label y under probability 1/(1+e^-z)
    p = 1.0 / (1.0 + math.exp(-z))
    return -(y * math.log(p) + (1.0 - y) * math.log(1.0 - p))


def pin_grad_at_zero():
    """At w = 0: linear gives -X_i^T y_i; logistic gives X_i^T (1/2 - y_i)."""
    for loss in ("linear", "logistic"):
        X, y = _tiny_regression(2, logistic=(loss == "logistic"))
        G = OG.chunk_gradients(X, y, np.zeros(X.shape[2]), loss)
        for i in range(X.shape[0]):
            want = -X[i].T @ y[i] if loss == "linear" else X[i].T @ (0.5 - y[i])
            assert np.allclose(G[i], want, rtol=1e-13, atol=1e-13)


def pin_grad_finite_difference():
    """Central differences of the summed per-sample loss match sum_i g_i (and each chunk alone)."""
    for loss in ("linear", "logistic"):
        X, y = _tiny_regression(3, logistic=(loss == "logistic"))
        w = rng(4).standard_normal(X.shape[2]) * 0.5
        G = OG.chunk_gradients(X, y, w, loss)
        h = 1e-6
        for i in range(X.shape[0]):
            for k in range(X.shape[2]):
                e = np.zeros_like(w)
                e[k] = h
                fp = sum(_sample_loss(X[i, r], y[i, r], w + e, loss) for r in range(X.shape[1]))
                fm = sum(_sample_loss(X[i, r], y[i, r], w - e, loss) for r in range(X.shape[1]))
                assert abs((fp - fm) / (2 * h) - G[i, k]) < 1e-6 * max(1.0, abs(G[i, k]))


def pin_grad_multi_point():
    X, y = _tiny_regression(5, logistic=True)
    W = rng(6).standard_normal((3, X.shape[2]))
    G = OG.chunk_gradients(X, y, W, "logistic")
    assert G.shape == (3, X.shape[0], X.shape[2])
    for q in range(3):
        for i in range(X.shape[0]):
            brute = np.zeros(X.shape[2])
            for r in range(X.shape[1]):
                z = float(X[i, r] @ W[q])
                brute += X[i, r] * (1.0 / (1.0 + math.exp(-z)) - y[i, r])
            assert np.allclose(G[q, i], brute, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# coverage, decodability, coefficients
# ---------------------------------------------------------------------------

def pin_fig1a_motivation():
    """Fig. 1(a): W3 failed, W1 slow (first chunk only); the full gradient is recoverable at
    ell = 1, while the original scheme (fully finished workers only) cannot cover D1."""
    O = OA.cyclic_O(3, 3, 1)
    psi = np.array([1, 2, 0])
    assert OP.decodable(O, psi, 1)
    assert OP.coverage(O, psi).tolist() == [1, 1, 1]
    finished = [j for j in range(3) if psi[j] == 2]
    covered = {i for j in finished for i in range(3) if O[i, j]}
    assert covered != {0, 1, 2}
    G = rng(7).standard_normal((3, 11))
    R = rng(8).standard_normal((1, 3))
    out = OP.run_pattern(O, psi, R, G)
    assert np.allclose(out["ghat"], G.sum(axis=0), rtol=1e-12, atol=1e-12)


def pin_sec2_2_support():
    O = sec2_2_O()
    exact = np.array(load_rows("sec2_2_support_exact.txt"), dtype=bool)
    approx = np.array(load_rows("sec2_2_support_approx.txt"), dtype=bool)
    assert (OP.indeterminate_support(O, np.array([5, 2, 0, 2, 3]), 2) == exact).all()
    assert (OP.indeterminate_support(O, np.array([4, 2, 0, 2, 3]), 2) == approx).all()
    assert OP.coverage(O, np.array([5, 2, 0, 2, 3])).tolist() == [3, 3, 2, 2, 2]
    assert OP.decodable(O, np.array([5, 2, 0, 2, 3]), 2)
    cov = OP.coverage(O, np.array([4, 2, 0, 2, 3]))
    assert cov[4] == 1 and not OP.decodable(O, np.array([4, 2, 0, 2, 3]), 2)
    assert OP.coef_err(O, np.array([4, 2, 0, 2, 3]), 2) == 1
    # the computed B has exactly the printed support (generic R: no indeterminate is zero)
    R = rng(9).standard_normal((2, 5))
    assert ((OP.encoding_matrix(O, np.array([5, 2, 0, 2, 3]), R) != 0) == exact).all()
    assert ((OP.encoding_matrix(O, np.array([4, 2, 0, 2, 3]), R) != 0) == approx).all()


def pin_sec2_2_closed_forms():
    """W5's system for the first column of B^(1): minimum-norm solution of
    [r01 r02 r05; r11 r12 r15][a1 b1 d1]^T = [1 0]^T is X^T (X X^T)^-1 e_0; and the
    over-determined 2x1 problem for d'_9, d'_10 of the approximate variant."""
    O = sec2_2_O()
    for seed in range(5):
        R = rng(100 + seed).standard_normal((2, 5))
        B = OP.encoding_matrix(O, np.array([5, 2, 0, 2, 3]), R)
        X = R[:, [0, 1, 4]]
        a, b, c = X[0] @ X[0], X[0] @ X[1], X[1] @ X[1]
        inv_col0 = np.array([c, -b]) / (a * c - b * b)          # (X X^T)^-1 e_0 via the adjugate
        want = X.T @ inv_col0
        assert np.allclose(B[[0, 1, 4], 0], want, rtol=1e-11, atol=1e-13)
        # W1, W2 and W5 all solve this problem and agree (Sec. 2.2)
        for beta in (0, 1, 4):
            sol = OP.worker_solve(beta, O, np.array([5, 2, 0, 2, 3]), R)
            got = [sol[(0, j, 0)] for j in (0, 1, 4)]
            assert np.allclose(got, want, rtol=1e-11, atol=1e-13)
        Bp = OP.encoding_matrix(O, np.array([4, 2, 0, 2, 3]), R)
        r05, r15 = R[0, 4], R[1, 4]
        den = r05 * r05 + r15 * r15
        assert np.isclose(Bp[4, 8], r05 / den, rtol=1e-12)
        assert np.isclose(Bp[4, 9], r15 / den, rtol=1e-12)


def _random_patterns(g, m, s, count):
    return [g.integers(0, s + 2, size=m) for _ in range(count)]


def pin_remark1_ell1():
    """ell = 1: the coefficient of W_j on D_i is R_j / sum_{j' in S_i} R_{j'}^2 (weighted partial sums)."""
    g = rng(10)
    for m, s in [(6, 2), (8, 3), (10, 1)]:
        O = OA.cyclic_O(m, m, s)
        for psi in _random_patterns(g, m, s, 10):
            R = g.standard_normal((1, m))
            B = OP.encoding_matrix(O, psi, R)
            for i in range(m):
                S = [j for j in range(m) if O[i, j] and O[i, j] <= psi[j]]
                den = sum(R[0, j] ** 2 for j in S)
                for j in range(m):
                    want = R[0, j] / den if j in S else 0.0
                    assert abs(B[j, i] - want) <= 1e-12 * max(1.0, abs(want))


def pin_ls_optimality():
    """Each B^(i) restricted to S_i satisfies the normal equations X^T (X b - e_k) = 0 and lies
    in the row space of X = R[:, S_i] (minimum norm)."""
    g = rng(11)
    for m, s, ell in [(6, 2, 2), (6, 2, 3), (8, 3, 4), (10, 4, 3)]:
        O = OA.cyclic_O(m, m, s)
        for psi in _random_patterns(g, m, s, 8):
            R = g.standard_normal((ell, m))
            B = OP.encoding_matrix(O, psi, R)
            for i in range(m):
                S = [j for j in range(m) if O[i, j] and O[i, j] <= psi[j]]
                others = [j for j in range(m) if j not in S]
                assert np.all(B[others, i * ell:(i + 1) * ell] == 0)
                if not S:
                    continue
                X = R[:, S]
                Bi = B[S, i * ell:(i + 1) * ell]
                assert np.abs(X.T @ (X @ Bi - np.eye(ell))).max() < 1e-10
                Q, _ = np.linalg.qr(X.T)            # orthonormal basis of range(X^T)
                Q = Q[:, :min(len(S), ell)]
                assert np.abs(Bi - Q @ (Q.T @ Bi)).max() < 1e-10


def pin_coef_err_identity():
    """|| 1^T (x) I - R B ||_F^2 of Algorithm 1's B equals sum_i max(0, ell - Delta_i) exactly
    (for an ell x Delta Gaussian X, ||X X^+ - I||_F^2 = ell - rank X; Sec. 2.1 sums it)."""
    g = rng(12)
    for m, s, ell in [(6, 2, 1), (6, 2, 2), (6, 2, 3), (8, 3, 4), (10, 2, 5)]:
        O = OA.cyclic_O(m, m, s)
        for psi in _random_patterns(g, m, s, 8):
            R = g.standard_normal((ell, m))
            B = OP.encoding_matrix(O, psi, R)
            assert abs(OP.coef_residual(B, R) - OP.coef_err(O, psi, ell)) < 1e-9


def _full_system_residual(O, psi, R):
    """Least-squares residual of R B = 1^T (x) I_ell over ALL indeterminates of B at once
    (the un-decoupled system): vec(R B) = (I (x) R) vec(B), columns restricted to the support."""
    ell, m = R.shape
    N = O.shape[0]
    support = np.repeat(((O != 0) & (O <= psi[None, :])).T, ell, axis=1)      # [m][N*ell]
    K = np.kron(np.eye(N * ell), R)
    cols = [c * m + j for c in range(N * ell) for j in range(m) if support[j, c]]
    target = np.tile(np.eye(ell), (1, N)).flatten(order="F")
    if not cols:
        return float(target @ target)
    A = K[:, cols]
    x = np.linalg.lstsq(A, target, rcond=None)[0]
    r = A @ x - target
    return float(r @ r)


BRUTE_CASES = [(3, 1), (4, 1), (5, 2), (6, 2)]


def pin_bruteforce_decodability(cases=BRUTE_CASES, ells=(1, 2, 3)):
    """Every psi in prod_j {0..delta}: full-system solvability <=> every Delta_i >= ell, and
    the full-system residual equals sum_i max(0, ell - Delta_i)."""
    for m, s in cases:
        O = OA.cyclic_O(m, m, s)
        for ell in ells:
            R = rng(1000 * m + 10 * s + ell).standard_normal((ell, m))
            for psi in itertools.product(range(s + 2), repeat=m):
                psi = np.array(psi)
                res = _full_system_residual(O, psi, R)
                assert (res <= 1e-9) == OP.decodable(O, psi, ell), (m, s, ell, psi)
                assert abs(res - OP.coef_err(O, psi, ell)) < 1e-8, (m, s, ell, psi)


def pin_worker_agreement():
    """Workers that processed the same chunk compute identical values for its indeterminates."""
    g = rng(13)
    for m, s, ell in [(6, 2, 2), (7, 3, 3)]:
        O = OA.cyclic_O(m, m, s)
        for psi in _random_patterns(g, m, s, 5):
            R = g.standard_normal((ell, m))
            sols = [OP.worker_solve(b, O, psi, R) for b in range(m)]
            merged = {}
            for sol in sols:
                for key, v in sol.items():
                    if key in merged:
                        assert abs(merged[key] - v) < 1e-12
                    merged[key] = v


def pin_two_routes():
    g = rng(14)
    for m, s, ell in [(6, 2, 1), (6, 2, 2), (8, 3, 3), (9, 2, 4)]:
        O = OA.cyclic_O(m, m, s)
        for psi in _random_patterns(g, m, s, 6):
            R = g.standard_normal((ell, m))
            G = g.standard_normal((m, 37))
            B = OP.encoding_matrix(O, psi, R)
            B2 = OP.encoding_matrix_per_chunk(O, psi, R)
            assert np.abs(B - B2).max() <= 1e-11 * max(1.0, np.abs(B2).max() ** 2)
            a = OP.reconstruct(OP.encode(B, G, ell), R, 37)
            b = OP.reconstruct_by_chunks(B, R, G)
            assert np.abs(a - b).max() < 1e-12 * max(1.0, np.abs(b).max())


def pin_mixing_projector():
    """What chunk i contributes to the estimate is M_i = R B^(i) applied to its blocks.  With B
    from the workers' own solves (Algorithm 1), M_i must be the orthogonal projector onto the
    range of R[:, S_i]: the identity once Delta_i >= ell (Gaussian R has full rank), zero when
    Delta_i = 0, and Q Q^T from a QR factorisation of R[:, S_i] in between (Sec. 2.1, Sec. 2.2)."""
    g = rng(19)
    for m, s, ell in [(6, 2, 2), (6, 2, 3), (8, 3, 3), (9, 2, 4), (7, 4, 5)]:
        O = OA.cyclic_O(m, m, s)
        for psi in _random_patterns(g, m, s, 8):
            R = g.standard_normal((ell, m))
            B = OP.encoding_matrix(O, psi, R)
            for i, S in enumerate(OP.processed_sets(O, psi)):
                M = R @ B[:, i * ell:(i + 1) * ell]
                if len(S) == 0:
                    ref = np.zeros((ell, ell))
                else:
                    Q, _ = np.linalg.qr(R[:, S])
                    Q = Q[:, :min(len(S), ell)]
                    ref = Q @ Q.T
                assert np.abs(M - ref).max() < 1e-9, (m, s, ell, psi, i)
                if len(S) >= ell:
                    assert np.abs(M - np.eye(ell)).max() < 1e-9


# ---------------------------------------------------------------------------
# encode + combine
# ---------------------------------------------------------------------------

def pin_exact_recovery():
    """No stragglers (psi = delta) and every ell <= s+1: the PS recovers sum_i g_i exactly;
    likewise for every decodable pattern, at any R.  Includes ell not dividing d (zero padding)."""
    g = rng(15)
    for m, s, d in [(6, 2, 64), (8, 3, 50), (5, 4, 33)]:
        O = OA.cyclic_O(m, m, s)
        G = g.standard_normal((m, d))
        want = G.sum(axis=0)
        for ell in range(1, s + 2):
            R = g.standard_normal((ell, m))
            out = OP.run_pattern(O, np.full(m, s + 1), R, G)
            assert out["dec"] and out["ghat"].shape == (d,)
            assert np.linalg.norm(out["ghat"] - want) <= 1e-12 * np.linalg.norm(want) * m
            for psi in _random_patterns(g, m, s, 12):
                if OP.decodable(O, psi, ell):
                    gh = OP.run_pattern(O, psi, R, G)["ghat"]
                    assert np.linalg.norm(gh - want) <= 1e-10 * np.linalg.norm(want)


def pin_ell1_masked_sum():
    """ell = 1, approximate: the estimate is the sum of the gradients of the covered chunks."""
    g = rng(16)
    for m, s in [(6, 2), (10, 3)]:
        O = OA.cyclic_O(m, m, s)
        G = g.standard_normal((m, 29))
        for psi in _random_patterns(g, m, s, 15):
            R = g.standard_normal((1, m))
            gh = OP.run_pattern(O, psi, R, G)["ghat"]
            cov = OP.coverage(O, psi)
            want = G[cov >= 1].sum(axis=0)
            assert np.abs(gh - want).max() < 1e-11 * max(1.0, np.abs(want).max())


def pin_mse_expectation(trials=1500):
    """Sec. 2.1: a chunk processed Delta < ell times has expected per-column error (ell - Delta)/ell
    over the randomness of R (Monte Carlo, 1500 draws of R; tolerance ~5 standard errors)."""
    m, s, ell = 8, 3, 4
    O = OA.cyclic_O(m, m, s)
    g = rng(17)
    # chunk 0 is held by workers 0, 7, 6, 5 at positions 1..4; these psi leave it Delta = 1, 2, 3
    for Delta, psi in [(1, [4, 4, 4, 4, 4, 3, 2, 1]), (2, [4, 4, 4, 4, 4, 3, 2, 4]), (3, [4, 4, 4, 4, 4, 3, 4, 4])]:
        psi = np.array(psi)
        assert OP.coverage(O, psi)[0] == Delta
        errs = np.zeros(ell)
        for _ in range(trials):
            R = g.standard_normal((ell, m))
            B = OP.encoding_matrix_per_chunk(O, psi, R)
            E = R @ B[:, 0:ell] - np.eye(ell)
            errs += (E ** 2).sum(axis=0)
        errs /= trials
        assert np.all(np.abs(errs - (ell - Delta) / ell) < 0.05), (Delta, errs)


def pin_compact_layout():
    """Bc[j][t][k] is the weight W_j gives block k of the t-th chunk in its order: encoding
    worker by worker from Bc over the processed prefix reproduces T = B G."""
    g = rng(18)
    for m, s, ell in [(6, 2, 1), (7, 3, 2), (8, 2, 3)]:
        O = OA.cyclic_O(m, m, s)
        order, _, _ = OA.tables(O)
        d = 31
        G = g.standard_normal((m, d))
        L = -(-d // ell)
        Gpad = np.zeros((m, ell * L))
        Gpad[:, :d] = G
        for psi in _random_patterns(g, m, s, 6):
            R = g.standard_normal((ell, m))
            B = OP.encoding_matrix(O, psi, R)
            Bc = OP.compact(B, O, ell)
            T = OP.encode(B, G, ell)
            for j in range(m):
                want = np.zeros(L)
                for t in range(psi[j]):
                    for k in range(ell):
                        want += Bc[j, t, k] * Gpad[order[j, t], k * L:(k + 1) * L]
                assert np.abs(T[j] - want).max() < 1e-12 * max(1.0, np.abs(want).max())
                assert np.all(Bc[j, psi[j]:] == 0)


def pin_widen_bf16():
    """bf16 storage: the stored 16 bits are the top half of an IEEE fp32 word (1 sign,
    8 exponent, 7 mantissa bits); widening is exact."""
    bits = np.array([0x3F80, 0xC000, 0x3F00, 0x0000, 0x8000, 0x4049, 0x7F7F, 0x0001], dtype=np.uint16)
    want = [1.0, -2.0, 0.5, 0.0, -0.0, 3.140625, 3.3895313892515355e38, 9.183549615799121e-41]
    got = OP.widen(bits, "bf16")
    assert got.dtype == np.float64 and list(got) == want
    assert np.signbit(got[4])
    f = np.array([1.5, -0.25], dtype=np.float32)
    assert list(OP.widen(f, "f32")) == [1.5, -0.25]


# ---------------------------------------------------------------------------
# Algorithm 2 (chunk ordering)
# ---------------------------------------------------------------------------

def _random_regular_support(g, m, delta):
    """Union of delta disjoint random permutation matrices (a delta-regular bipartite support)."""
    while True:
        S = np.zeros((m, m), dtype=bool)
        ok = True
        for _ in range(delta):
            for _try in range(200):
                perm = g.permutation(m)
                if not S[np.arange(m), perm].any():
                    S[np.arange(m), perm] = True
                    break
            else:
                ok = False
                break
        if ok:
            return S


def check_ordering(O, S):
    """O is an ordering of support S whose every row sums to delta(delta+1)/2 (Sec. 3 optimum)."""
    O = np.asarray(O)
    delta = int(S.sum(axis=0)[0])
    assert ((O != 0) == S).all()
    for j in range(O.shape[1]):
        assert sorted(O[S[:, j], j].tolist()) == list(range(1, delta + 1))
    assert (O.sum(axis=1) == delta * (delta + 1) // 2).all()
    assert OO.q_max(O) == delta * (delta + 1) // 2 + (O.shape[1] - delta - 1) * delta


def pin_ordering_bruteforce_optimum():
    """On tiny regular supports, Algorithm 2 reaches the minimum Q_max over every ordering
    (each column's delta! orders enumerated)."""
    g = rng(30)
    for m, delta in [(4, 2), (5, 2), (4, 3), (5, 3)]:
        S = _random_regular_support(g, m, delta)
        per_col = []
        for j in range(m):
            rows = np.flatnonzero(S[:, j])
            per_col.append([dict(zip(rows, perm)) for perm in itertools.permutations(range(1, delta + 1))])
        best = None
        for choice in itertools.product(*per_col):
            O = np.zeros((m, m), dtype=np.int64)
            for j, mp in enumerate(choice):
                for i, v in mp.items():
                    O[i, j] = v
            qm = int(OA.Q(O).max())
            best = qm if best is None else min(best, qm)
        O = OO.chunk_ordering(S)
        check_ordering(O, S)
        assert OO.q_max(O) == best


def pin_ordering_regular_graphs():
    """Random regular supports and a random regular graph's adjacency: valid, optimal orderings;
    the cyclic support gets the same Q_max as the cyclic order."""
    g = rng(31)
    for m, delta in [(10, 3), (50, 5), (64, 8)]:
        S = _random_regular_support(g, m, delta)
        check_ordering(OO.chunk_ordering(S), S)
    from workloads import gen
    A = gen.random_regular_graph(60, 6) != 0
    check_ordering(OO.chunk_ordering(A), A)
    C = OA.cyclic_O(12, 12, 3)
    assert OO.q_max(OO.chunk_ordering(C != 0)) == OO.q_max(C)


# ---------------------------------------------------------------------------
# simulation (Sec. 4)
# ---------------------------------------------------------------------------

def pin_simulation_hand_example():
    """Fig. 1(a)'s system (W_i holds D_i then D_{i+1}) with chunk times worked by hand:
    W1: 1, 3 (finishes D1 at 1, D2 at 4); W2: 2, 2 (D2 at 2, D3 at 4); W3 failed.
    ell = 1: D1 at 1, D2 at 2, D3 at 4 -> the protocol completes at 4; original GC needs
    finished workers covering D1..D3: W1 (done at 4) covers D1, D2, W2 (done at 4) D2, D3 -> 4.
    ell = 2: D1's copies are on W1 and W3 (failed) -> never."""
    O = OA.cyclic_O(3, 3, 1)
    tau = np.array([[[1.0, 3.0], [2.0, 2.0], [5.0, 5.0]]])
    failed = np.array([[False, False, True]])
    part, orig = OS.completion_times(tau, failed, O, 1)
    assert part[0] == 4.0 and orig[0] == 4.0
    part2, orig2 = OS.completion_times(tau, failed, O, 2)
    assert np.isinf(part2[0]) and np.isinf(orig2[0])
    tau_b = np.array([[[1.0, 3.0], [2.0, 2.0], [0.5, 9.0]]])       # W3 alive: D3 at 0.5
    part, orig = OS.completion_times(tau_b, None, O, 1)
    assert part[0] == 2.0 and orig[0] == 4.0                       # original waits for W1 or W2 to finish
    psi = OS.progress(tau, failed, np.array([0.5, 1.0, 3.9, 4.0]))
    assert psi[0].tolist() == [[0, 0, 0], [1, 0, 0], [1, 1, 0], [2, 2, 0]]


def pin_simulation_grid_route():
    """Second route: at every event time T (the only times the state changes), decide
    decodability of psi(T) with the protocol's coverage; the first decodable one is the
    completion time.  Original GC: psi_j = delta once worker j is done, else 0."""
    g = rng(40)
    for m, s, ell, nfail in [(6, 2, 1, 1), (8, 3, 2, 1), (10, 3, 3, 1), (7, 2, 1, 0)]:
        O = OA.cyclic_O(m, m, s)
        for _ in range(6):
            tau = g.exponential(1.0, size=(1, m, s + 1))
            failed = np.zeros((1, m), dtype=bool)
            failed[0, g.choice(m, nfail, replace=False)] = True
            part, orig = OS.completion_times(tau, failed, O, ell)
            cum = np.cumsum(tau[0], axis=1)
            times = np.unique(cum[~failed[0]].ravel())
            psi_all = OS.progress(tau, failed, times)[0]
            dec = [OP.decodable(O, psi_all[k], ell) for k in range(len(times))]
            want = times[dec.index(True)] if any(dec) else np.inf
            assert part[0] == want
            fulls = np.unique(cum[~failed[0], -1])
            dec_o = [OP.decodable(O, np.where((cum[:, -1] <= T) & ~failed[0], s + 1, 0), ell) for T in fulls]
            want_o = fulls[dec_o.index(True)] if any(dec_o) else np.inf
            assert orig[0] == want_o
            assert part[0] <= orig[0]


def pin_original_ls():
    """Original GC's least-squares error: closed forms and a projection identity.
    No finished worker: N.  One finished worker of load delta: N - delta.  Finished workers
    whose supports partition the chunks: 0.  In general ||(I - Q Q^T) 1||^2 for an
    orthonormal basis Q of range(A_F) (QR, a different routine than the oracle's lstsq)."""
    O = OA.cyclic_O(6, 6, 1)                      # worker j holds chunks j, j+1
    assert OS.original_ls_error(O, np.zeros(6)) == 6.0
    assert abs(OS.original_ls_error(O, np.array([2, 0, 0, 0, 0, 0])) - 4.0) < 1e-12
    assert abs(OS.original_ls_error(O, np.array([2, 0, 2, 0, 2, 0]))) < 1e-12   # {0,1},{2,3},{4,5}
    g = rng(41)
    from workloads import gen
    A = gen.random_regular_graph(30, 4) != 0
    O2 = OO.chunk_ordering(A)
    for _ in range(20):
        psi = g.integers(0, 5, size=30)
        F = np.flatnonzero(psi >= 4)
        want = 30.0
        if len(F):
            Q, Rr = np.linalg.qr(A[:, F].astype(float))
            keep = np.abs(np.diag(Rr)) > 1e-10
            Q = Q[:, keep]
            v = np.ones(30) - Q @ (Q.T @ np.ones(30))
            want = float(v @ v)
        assert abs(OS.original_ls_error(O2, psi) - want) < 1e-9


ALL_PINS = [
    pin_fig1a_ordering, pin_cyclic_invariants, pin_tables_roundtrip,
    pin_grad_at_zero, pin_grad_finite_difference, pin_grad_multi_point,
    pin_fig1a_motivation, pin_sec2_2_support, pin_sec2_2_closed_forms, pin_remark1_ell1,
    pin_ls_optimality, pin_coef_err_identity, pin_worker_agreement, pin_two_routes,
    pin_mixing_projector,
    pin_exact_recovery, pin_ell1_masked_sum, pin_compact_layout, pin_widen_bf16,
    pin_ordering_bruteforce_optimum, pin_ordering_regular_graphs,
    pin_simulation_hand_example, pin_simulation_grid_route, pin_original_ls,
]
