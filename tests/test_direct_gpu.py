"""GPU parity of gc_decode_direct: the estimate formed from the chunk gradients through the
per-chunk mixing matrices M_i = R[:, S_i] pinv(R[:, S_i]) (Sec. 2, Sec. 2.2), against the oracle.

Elementwise bound: one fp32 rounding of each M_i entry plus the fp32 sum over N*ell terms
(gamma_{N ell + 2} times sum_i |M_i| |g_i|), plus the fp64 Gram/Cholesky error of M_i where
0 < Delta_i < ell (about kappa^2 2^-53 relative).  Exact patterns have M_i in {0, I}, so there
the GPU result is an fp32 sum of the covered chunks.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle.assignment as OA
import oracle.protocol as OP
import oracle_runs as R_
from workloads import HEADLINE, SMALL, TINY, Workload, gen

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2405_19509_amd import gcx  # noqa: E402


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def tables(wl):
    O, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_CYCLIC, wl.N, wl.m, wl.s)
    return O.astype(np.int64), order, holder, hpos


def run_direct(wl, G, psi, ell, dtype="f32", want_ghat=True):
    O, order, holder, hpos = tables(wl)
    R = gen.shared_R(wl.m, ell)
    Gd = dev(G) if dtype == "f32" else dev(G.view(np.int16)).view(torch.bfloat16)
    gsum = gcx.gc_sum_chunks(Gd)
    ghat, sqerr = gcx.gc_decode_direct(Gd, dev(psi), dev(order), dev(holder), dev(hpos), dev(R),
                                       gsum=gsum, want_ghat=want_ghat)
    return O, R, ghat, sqerr, gsum


def check_elementwise(O, psi, R, G64, gh, label):
    ell = R.shape[0]
    K = O.shape[0] * ell
    ref, mag, kap = R_.direct_ref(O, psi, R, G64)
    magG = np.abs(R_.gblocks(G64, ell)).sum(axis=(0, 1)).reshape(1, -1)         # [1][L]
    magG = np.tile(magG, (1, ell))[:, :G64.shape[1]]
    bound = 2 * R_.gamma(K + 2) * mag + 1e-13 * (kap ** 2)[:, None] * magG
    err = np.abs(gh - ref)
    assert (err <= bound + 1e-30).all(), (label, float((err / (bound + 1e-30)).max()))
    return ref, kap


@pytest.mark.parametrize("ell", [1, 2, 3])
def test_direct_tiny_every_pattern(ell):
    """m = 6, d = 64, all 100 patterns: estimate and squared error against the oracle."""
    wl = TINY
    X, y, w = gen.regression_data(wl)
    G64 = R_.chunk_grads(X, y, w, wl.loss)
    G = G64.astype(np.float32)
    psi = gen.psi(wl)
    O, R, ghat, sqerr, gsum = run_direct(wl, G, psi, ell)
    ref, _ = check_elementwise(O, psi, R, G.astype(np.float64), host(ghat).astype(np.float64), "tiny")
    # the same estimate through the protocol's own route (Algorithm 1 at every worker)
    e2e = R_.end_to_end(O, psi, R, G.astype(np.float64), per_worker=True)
    assert np.abs(e2e - ref).max() <= 1e-9 * max(1.0, np.abs(ref).max())
    tgt = G.astype(np.float64).sum(axis=0)
    se_ref = ((ref - tgt) ** 2).sum(axis=1)
    se = host(sqerr)
    se_gh = ((host(ghat).astype(np.float64) - host(gsum).astype(np.float64)) ** 2).sum(axis=1)
    assert (np.abs(se - se_gh) <= 8 * R_.U * se_gh + 1e-30).all()
    scale = float((np.abs(G.astype(np.float64)).sum(axis=0) ** 2).sum())
    assert (np.abs(se - se_ref) <= 1e-5 * scale).all()
    # at ell = 1 the 100 patterns hold both decodable and non-decodable ones
    dec = np.array([OP.decodable(O, p, ell) for p in psi])
    assert (~dec).any() and (dec.any() or ell > 1)


@pytest.mark.parametrize("ell", [1, 2])
def test_direct_small_spans_tiles(ell):
    """m = 20, d = 4096, 1,000 patterns (8 row tiles at ell = 1, 32 column tiles): every pattern
    elementwise, rel-L2 <= 1e-5 where the mixing blocks are well conditioned."""
    wl = SMALL
    X, y, w = gen.regression_data(wl)
    G = R_.chunk_grads(X, y, w, wl.loss).astype(np.float32)
    psi = gen.psi(wl)
    O, R, ghat, sqerr, _ = run_direct(wl, G, psi, ell)
    gh = host(ghat).astype(np.float64)
    pats = np.arange(0, wl.P, 7)
    ref, kap = check_elementwise(O, psi[pats], R, G.astype(np.float64), gh[pats], "small")
    rel = np.linalg.norm(gh[pats] - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-300)
    assert rel[kap <= 100].max(initial=0.0) <= 1e-5


@pytest.mark.parametrize("N,d,ell,dtype", [
    (37, 1001, 3, "f32"),     # K = 111 (ragged last k stage), d % 4 != 0, L = 334 (ragged tile)
    (20, 1000, 8, "f32"),     # d % ell != 0: zero-padded last block
    (23, 2050, 2, "bf16"),    # bf16 gradients, vector loads
    (11, 999, 1, "bf16"),     # bf16, scalar loads
])
def test_direct_ragged(N, d, ell, dtype):
    wl = Workload(name=f"ragged_m{N}_d{d}", N=N, m=N, s=min(N - 1, max(ell, 3)), d=d, P=300,
                  ells=(ell,), g_dtype=dtype, pattern="uniform")
    G = gen.given_G(wl)
    psi = gen.psi(wl)
    psi[::10] = wl.delta                     # every tenth pattern: no stragglers (exact)
    G64 = OP.widen(G, dtype)
    O, R, ghat, sqerr, gsum = run_direct(wl, G, psi, ell, dtype)
    gh = host(ghat).astype(np.float64)
    ref, _ = check_elementwise(O, psi, R, G64, gh, wl.name)
    # squared errors: those of the returned estimate (fp32 differences and squares: relative
    # 6 * 2^-24), and the oracle's up to the estimate's own error
    se = host(sqerr)
    tgt32 = host(gsum).astype(np.float64)
    se_gh = ((gh - tgt32) ** 2).sum(axis=1)
    assert (np.abs(se - se_gh) <= 8 * R_.U * se_gh + 1e-30).all()
    se_ref = ((ref - G64.sum(axis=0)) ** 2).sum(axis=1)
    scale = float((np.abs(G64).sum(axis=0) ** 2).sum())
    assert (np.abs(se - se_ref) <= 1e-5 * scale).all()
    # error-only mode gives the same squared errors, bit for bit
    _, _, g2, se2, _ = run_direct(wl, G, psi, ell, dtype, want_ghat=False)
    assert g2 is None and np.array_equal(host(se2), host(sqerr))


def test_direct_single_pattern_and_no_stragglers():
    """P = 1 and psi = delta (everything processed): the estimate is the exact sum."""
    wl = Workload(name="full_m9_d300", N=9, m=9, s=2, d=300, P=1, ells=(3,))
    G = gen.given_G(wl)
    psi = np.full((1, 9), 3, dtype=np.int32)
    for ell in (1, 2, 3):
        O, R, ghat, sqerr, gsum = run_direct(wl, G, psi, ell)
        tgt = G.astype(np.float64).sum(axis=0)
        assert np.abs(host(ghat)[0] - tgt).max() <= R_.gamma(9 * ell + 2) * np.abs(G).sum(axis=0).max()
        assert host(sqerr)[0] <= 1e-10 * (tgt ** 2).sum()


@pytest.fixture(scope="module")
def headline_G():
    X, y, w = gen.regression_data(HEADLINE)
    return R_.chunk_grads(X, y, w, HEADLINE.loss)


@pytest.mark.parametrize("ell", [1, 2])
def test_direct_headline_full_size(headline_G, ell):
    """m = 50, d = 16384, all 10,000 patterns, the bench's call: squared errors of every pattern
    (ell = 1: against ||sum of uncovered chunks||^2) and the full estimate on sampled patterns."""
    wl = HEADLINE
    G64 = headline_G
    G = G64.astype(np.float32)
    psi = gen.psi(wl)
    O, R, ghat, sqerr, _ = run_direct(wl, G, psi, ell)
    G64 = G.astype(np.float64)
    pats = list(range(0, wl.P, wl.P // 25)) + [wl.P - 1]
    gh = host(ghat[torch.as_tensor(pats, device="cuda")]).astype(np.float64)
    ref, kap = check_elementwise(O, psi[pats], R, G64, gh, "headline")
    rel = np.linalg.norm(gh - ref, axis=1) / np.linalg.norm(ref, axis=1)
    assert rel[kap <= 100].max(initial=0.0) <= 1e-5
    se = host(sqerr)
    tgt = G64.sum(axis=0)
    if ell == 1:
        cov = np.stack([OP.coverage(O, p) for p in psi])
        miss = (cov == 0).astype(np.float64) @ G64
        se_ref = (miss ** 2).sum(axis=1)
    else:
        se_ref = ((ref - tgt) ** 2).sum(axis=1)
        se = se[pats]
    scale = np.linalg.norm(tgt)
    assert (np.abs(np.sqrt(se) - np.sqrt(se_ref)) <= 1e-5 * scale + 1e-4 * np.sqrt(se_ref)).all()


def check_sampled_direct(O, psi, R, G, dtype, ghat_d, pats, xs):
    """The estimate at positions k*L + xs of patterns pats against the oracle's
    sum_i M_i g_i computed on just those positions (``oracle_runs.sampled_blocks``)."""
    ell = R.shape[0]
    d = G.shape[1]
    L = -(-d // ell)
    Gsub = R_.sampled_blocks(G, dtype, ell, xs)                 # blocks of width len(xs)
    cols = [k * L + int(x) for k in range(ell) for x in xs]
    keep = [a for a, c in enumerate(cols) if c < d]
    idx = torch.as_tensor([cols[a] for a in keep], device="cuda")
    ref, mag, kap = R_.direct_ref(O, psi[pats], R, Gsub)         # [len(pats)][ell*len(xs)]
    magG = np.tile(np.abs(R_.gblocks(Gsub, ell)).sum(axis=(0, 1)), ell)
    K = O.shape[0] * ell
    for a, p in enumerate(pats):
        gh = host(ghat_d[p][idx]).astype(np.float64)
        bound = 2 * R_.gamma(K + 2) * mag[a][keep] + 1e-13 * kap[a] ** 2 * magG[keep]
        assert (np.abs(gh - ref[a][keep]) <= bound + 1e-30).all(), (p, np.abs(gh - ref[a][keep]).max())


def test_direct_bandwidth_full_size():
    """m = 100, d = 2^20, fp32 gradients: 12 patterns at ell = 1, 2, 8 (K up to 800 through the
    k-staged kernel, 8,192 column tiles at ell = 1), sampled positions against the oracle."""
    from workloads import BANDWIDTH
    wl = BANDWIDTH
    O, order, holder, hpos = tables(wl)
    psi = gen.psi(wl, count=12)
    psi[5] = 0                                   # nothing processed: estimate zero
    G = gen.given_G(wl, threads=16)
    Gd = dev(G)
    gsum = gcx.gc_sum_chunks(Gd)
    for ell in (1, 2, 8):
        R = gen.shared_R(wl.m, ell)
        ghat, sqerr = gcx.gc_decode_direct(Gd, dev(psi), dev(order), dev(holder), dev(hpos), dev(R),
                                           gsum=gsum)
        L = -(-wl.d // ell)
        xs = np.sort(np.random.default_rng(30 + ell).choice(L, 48, replace=False))
        check_sampled_direct(O, psi, R, G, "f32", ghat, [0, 3, 5, 11], xs)
        assert float(host(ghat[5]).__abs__().max()) == 0.0
        tgt = host(gsum).astype(np.float64)
        assert abs(host(sqerr)[5] - (tgt ** 2).sum()) <= 1e-5 * (tgt ** 2).sum()
        del ghat
        torch.cuda.empty_cache()


def test_direct_large_bf16_full_length():
    """m = 200, d = 2^24, bf16 gradients, least-squares patterns (50% forced stragglers):
    two patterns at full length for ell = 1, 2, 4, sampled positions against the oracle."""
    from workloads import LARGE
    wl = LARGE
    O, order, holder, hpos = tables(wl)
    psi = gen.psi(wl, count=2, variant="ls")
    G = gen.given_G(wl, threads=16)
    Gd = dev(G.view(np.int16)).view(torch.bfloat16)
    gsum = gcx.gc_sum_chunks(Gd)
    for ell in (1, 2, 4):
        R = gen.shared_R(wl.m, ell)
        ghat, sqerr = gcx.gc_decode_direct(Gd, dev(psi), dev(order), dev(holder), dev(hpos), dev(R),
                                           gsum=gsum)
        L = -(-wl.d // ell)
        xs = np.sort(np.random.default_rng(40 + ell).choice(L, 24, replace=False))
        check_sampled_direct(O, psi, R, G, "bf16", ghat, [0, 1], xs)
        # the squared error agrees with the estimate it comes with
        gh = host(ghat).astype(np.float64)
        se_gh = ((gh - host(gsum).astype(np.float64)) ** 2).sum(axis=1)
        assert (np.abs(host(sqerr) - se_gh) <= 8 * R_.U * se_gh).all()
        del ghat, gh
        torch.cuda.empty_cache()
