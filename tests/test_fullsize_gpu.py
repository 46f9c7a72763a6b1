"""GPU parity at the workloads' full sizes, in the launch configuration bench.py times.

Integer outputs are compared with the oracle for every pattern.  Floating-point
outputs are compared on sampled patterns and sampled positions that the oracle
computes one by one (``oracle_runs.sampled_blocks``), and through properties
that hold at any size (at ell = 1 the squared error of every pattern is
||sum of the uncovered chunks' gradients||^2).
"""
from __future__ import annotations

import os

import numpy as np
import pytest

import oracle.assignment as OA
import oracle.protocol as OP
import oracle_runs as R_
from workloads import BANDWIDTH, HEADLINE, LARGE, gen

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2405_19509_amd import gcx  # noqa: E402

U = R_.U
THREADS = min(16, len(os.sched_getaffinity(0)))


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def tables(wl):
    O, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_CYCLIC, wl.N, wl.m, wl.s)
    return O.astype(np.int64), order, holder, hpos


def check_integers(O, psi, ell, cov, dec, cerr):
    for p in range(len(psi)):
        c = OP.coverage(O, psi[p])
        assert (cov[p] == c).all(), p
        assert dec[p] == int((c >= ell).all()), p
        assert cerr[p] == int(np.maximum(0, ell - c).sum()), p


def check_sampled(O, order, psi, R, G, dtype, T_d, ghat_d, pats, xs, ell):
    """T[p][j][xs] and the estimate at k*L + xs for patterns pats, against the oracle."""
    d = G.shape[1]
    L = -(-d // ell)
    Gsub = R_.sampled_blocks(G, dtype, ell, xs)
    xs_t = torch.as_tensor(np.asarray(xs), device="cuda")
    delta = order.shape[1]
    Rd = R.astype(np.float64)
    for p in pats:
        B = OP.encoding_matrix_per_chunk(O, psi[p], R)
        kap = max([np.linalg.cond(Rd[:, S]) for S in OP.processed_sets(O, psi[p]) if len(S)] + [1.0])
        T_ref = OP.encode(B, Gsub, ell)                                  # [m][S]
        gh_ref = Rd @ T_ref                                              # [ell][S]
        T = host(T_d[p][:, xs_t]).astype(np.float64)
        sent = psi[p] > 0
        # sum of |terms| of each T entry; its error: fp32 rounding of the coefficients and the
        # delta*ell-term fp32 sum (for bf16 gradients the matrix cores' split-coefficient sum),
        # plus the fp64 Gram/Cholesky solve (~kappa^2 2^-53)
        Mag = OP.encode(np.abs(B), np.abs(Gsub), ell)
        eps_T = max(2 * R_.gamma(ell * delta + 2), R_.encode_eps(ell * delta, dtype) + 2 * U) + 1e-14 * kap ** 2
        assert (np.abs(T[sent] - T_ref[sent]) <= eps_T * Mag[sent] + 1e-30).all(), p
        if ghat_d is not None:
            cols = [k * L + x for k in range(ell) for x in xs]
            keep = [a for a, c in enumerate(cols) if c < d]
            gh = host(ghat_d[p][torch.as_tensor([cols[a] for a in keep], device="cuda")]).astype(np.float64)
            ref = gh_ref.reshape(-1)[keep]
            mag_T = (np.abs(Rd) @ np.abs(T_ref)).reshape(-1)[keep]
            mag_G = (np.abs(Rd) @ Mag).reshape(-1)[keep]
            bound = 2 * R_.gamma(O.shape[1] + 2) * mag_T + eps_T * mag_G
            assert (np.abs(gh - ref) <= bound + 1e-30).all(), p


@pytest.mark.parametrize("ell", [1, 2])
def test_headline_full_size(ell):
    """m = 50, d = 16384, n = 512, all 10,000 patterns: the bench's calls and launch shapes."""
    wl = HEADLINE
    O, order, holder, hpos = tables(wl)
    X, y, w = gen.regression_data(wl)
    psi = gen.psi(wl)
    R = gen.shared_R(wl.m, ell)
    P = wl.P
    L = -(-wl.d // ell)
    G = gcx.gc_chunk_grads(dev(X), dev(y), dev(w), gcx.GC_LOSS_LOGISTIC)
    gsum = gcx.gc_sum_chunks(G)
    psid = dev(psi)
    cov, dec, cerr, Bc = gcx.gc_decode_coeffs(psid, dev(order), dev(holder), dev(hpos), dev(R))
    T = gcx.gc_encode(G, psid, dev(order), Bc)
    ghat, sqerr = gcx.gc_reconstruct(T, dev(R), wl.d, psi=psid, gsum=gsum)
    assert T.shape == (P, wl.m, L)

    G_ref = R_.chunk_grads(X, y, w, wl.loss)
    del X
    Gh = host(G).astype(np.float64)
    rel = np.linalg.norm(Gh - G_ref, axis=1) / np.linalg.norm(G_ref, axis=1)
    assert rel.max() <= 1e-5
    check_integers(O, psi, ell, host(cov), host(dec), host(cerr))

    pats = list(range(0, P, P // 12)) + [P - 1]
    Bc_ref, kappa = R_.coefficients(O, psi[pats], R)
    Bc_s = host(Bc[torch.as_tensor(pats, device="cuda")]).astype(np.float64)
    assert (np.abs(Bc_s - Bc_ref) <= R_.bc_bound(Bc_ref, kappa, O)).all()
    # the whole estimate on the sampled patterns, from the oracle's own fp64 gradients
    gh_ref = R_.end_to_end(O, psi[pats], R, G_ref)
    gh = host(ghat[torch.as_tensor(pats, device="cuda")]).astype(np.float64)
    rel = np.linalg.norm(gh - gh_ref, axis=1) / np.linalg.norm(gh_ref, axis=1)
    if ell == 1:
        assert rel.max() <= 1e-5, rel.max()
    else:
        well = kappa.max(axis=1) <= 100
        print(f"ell={ell}: rel-L2 {rel.max():.2e} (max), {rel[well].max(initial=0.0):.2e} over "
              f"{int(well.sum())}/{len(pats)} sampled patterns with kappa <= 100")
        assert rel[well].max(initial=0.0) <= 1e-5, rel
    # T at sampled positions on identical inputs: the encode re-run on the oracle's gradients
    # rounded to fp32 (the pipeline above fed it the GPU's own gradients)
    G32 = G_ref.astype(np.float32)
    T = gcx.gc_encode(dev(G32), psid, dev(order), Bc, T=T)
    check_sampled(O, order, psi, R, G32, "f32", T, None, pats[:4],
                  np.random.default_rng(ell).choice(L, 48, replace=False), ell)

    if ell == 1:
        # every pattern: the estimate is the sum of the covered chunks, so the squared error
        # is the squared norm of the sum of the uncovered ones
        covh = host(cov)
        miss = (covh == 0).astype(np.float64) @ G_ref                      # [P][d]
        se_ref = (miss ** 2).sum(axis=1)
        se = host(sqerr)
        scale = np.linalg.norm(G_ref.sum(axis=0))
        assert (np.abs(np.sqrt(se) - np.sqrt(se_ref)) <= 1e-5 * scale + 1e-4 * np.sqrt(se_ref)).all()


def test_bandwidth_full_size():
    """m = 100, d = 2^20: coefficients for all 10,000 patterns; encode + combine on a batch."""
    wl = BANDWIDTH
    O, order, holder, hpos = tables(wl)
    psi = gen.psi(wl)
    G = gen.given_G(wl, threads=THREADS)
    Gd = dev(G)
    gsum = gcx.gc_sum_chunks(Gd)
    batch = 12
    for ell in (1, 2, 8):
        R = gen.shared_R(wl.m, ell)
        cov, dec, cerr, Bc = gcx.gc_decode_coeffs(dev(psi), dev(order), dev(holder), dev(hpos), dev(R))
        check_integers(O, psi, ell, host(cov), host(dec), host(cerr))
        if ell <= 6:
            assert (host(dec) == 1).all()        # this straggler model always leaves >= 7 copies
        pb = dev(psi[:batch])
        T = gcx.gc_encode(Gd, pb, dev(order), Bc[:batch].contiguous())
        ghat, sqerr = gcx.gc_reconstruct(T, dev(R), wl.d, psi=pb, gsum=gsum)
        L = -(-wl.d // ell)
        check_sampled(O, order, psi, R, G, "f32", T, ghat, range(0, batch, 3),
                      np.random.default_rng(10 + ell).choice(L, 64, replace=False), ell)
        se = host(sqerr)
        decs = host(dec)[:batch] == 1
        scale = float((G.astype(np.float64).sum(axis=0) ** 2).sum())
        assert (se[decs] <= 1e-8 * scale).all()
        del T, ghat
        torch.cuda.empty_cache()


@pytest.mark.parametrize("variant,ells", [("exact", (1, 2)), ("ls", (1, 2, 4))])
def test_large_full_size(variant, ells):
    """m = 200, d = 2^24, bf16 chunk gradients: coefficients for all 100,000 patterns in one
    call (integers for every pattern, Bc on sampled patterns); encode + combine for single
    patterns at full length (13.4 GB of T at ell = 1)."""
    wl = LARGE
    O, order, holder, hpos = tables(wl)
    psi = gen.psi(wl, variant=variant)
    P = len(psi)
    # coefficient rows checked against the oracle: the first patterns, both sides of the
    # waves' first and later passes over the batch, and the last ones
    rng = np.random.default_rng(31)
    sample = sorted(set([0, 1, 2, 63, 64, 4095, 4096, 8191, 8192, 8193, 16383, 16384, P // 2,
                         P - 2, P - 1] + rng.choice(P, 9, replace=False).tolist()))
    sample_t = torch.as_tensor(sample, device="cuda")
    for ell in ells:
        R = gen.shared_R(wl.m, ell)
        cov, dec, cerr, Bc = gcx.gc_decode_coeffs(dev(psi), dev(order), dev(holder), dev(hpos), dev(R))
        Bc_s = host(Bc[sample_t])
        del Bc
        cov, dec, cerr = host(cov), host(dec), host(cerr)
        Bc_ref, kappa = R_.coefficients(O, psi[sample], R)
        bound = R_.bc_bound(Bc_ref, kappa, O)
        diff = np.abs(Bc_s.astype(np.float64) - Bc_ref)
        worst = np.unravel_index(np.argmax(diff - bound), diff.shape)
        assert (diff <= bound).all(), f"Bc off at pattern {sample[worst[0]]}, {worst[1:]}"
        # all 100,000 patterns: coverage against the oracle's definition, vectorised over patterns
        ref = np.zeros_like(cov)
        for t in range(wl.delta):
            # worker (i - t) mod N holds chunk i at position t
            ref += psi[:, (np.arange(wl.N) - t) % wl.m] > t
        assert (cov == ref).all()
        assert (dec == (ref >= ell).all(axis=1)).all()
        assert (cerr == np.maximum(0, ell - ref).sum(axis=1)).all()
        check_integers(O, psi[:200], ell, cov[:200], dec[:200], cerr[:200])
    G = gen.given_G(wl, threads=THREADS)
    Gd = dev(G.view(np.int16)).view(torch.bfloat16)
    gsum = gcx.gc_sum_chunks(Gd)
    ell = ells[-1]
    R = gen.shared_R(wl.m, ell)
    p0 = 1
    pb = dev(psi[p0:p0 + 1])
    _, _, _, Bc = gcx.gc_decode_coeffs(pb, dev(order), dev(holder), dev(hpos), dev(R))
    T = gcx.gc_encode(Gd, pb, dev(order), Bc)
    ghat, sqerr = gcx.gc_reconstruct(T, dev(R), wl.d, psi=pb, gsum=gsum)
    L = -(-wl.d // ell)
    check_sampled(O, order, psi[p0:p0 + 1], R, G, "bf16", T, ghat, [0],
                  np.random.default_rng(20 + ell).choice(L, 48, replace=False), ell)
    assert np.isfinite(host(sqerr)).all()


_LARGE_G = {}


def _large_G():
    if "G" not in _LARGE_G:
        _LARGE_G["G"] = gen.given_G(LARGE, threads=THREADS)
    return _LARGE_G["G"]


@pytest.mark.parametrize("variant,ell,per_call", [("exact", 1, 16), ("exact", 2, 32), ("ls", 1, 16),
                                                  ("ls", 2, 32), ("ls", 4, 64)])
def test_large_encode_bench_launch(variant, ell, per_call):
    """m = 200, d = 2^24, bf16 chunk gradients: the first call of each of the bench's configs
    rows (16 / 32 / 64 patterns per call: 64- and 128-candidate windows, runs of 32 slices,
    T up to 215 GB), T and the estimate on sampled patterns and positions (slice and run
    boundaries among them)."""
    wl = LARGE
    O, order, holder, hpos = tables(wl)
    psi = gen.psi(wl, count=per_call, variant=variant)
    R = gen.shared_R(wl.m, ell)
    G = _large_G()
    Gd = dev(G.view(np.int16)).view(torch.bfloat16)
    pd = dev(psi)
    _, _, _, Bc = gcx.gc_decode_coeffs(pd, dev(order), dev(holder), dev(hpos), dev(R))
    T = gcx.gc_encode(Gd, pd, dev(order), Bc)
    ghat, sqerr = gcx.gc_reconstruct(T, dev(R), wl.d, psi=pd, gsum=gcx.gc_sum_chunks(Gd))
    L = -(-wl.d // ell)
    rng = np.random.default_rng(50 + ell)
    xs = sorted(set([0, 255, 256, 511, 512, 8191, 8192, L - 257, L - 1] + rng.choice(L, 40, replace=False).tolist()))
    pats = sorted(set([0, per_call // 2, per_call - 1]))
    check_sampled(O, order, psi, R, G, "bf16", T, ghat, pats, xs, ell)
    assert np.isfinite(host(sqerr)).all()
    del T, ghat, Bc, Gd
    torch.cuda.empty_cache()


@pytest.mark.parametrize("ell,per_call", [(1, 256), (2, 512), (8, 1024)])
def test_bandwidth_encode_bench_launch(ell, per_call):
    """m = 100, d = 2^20, fp32 chunk gradients: the first call of each of the bench's configs
    rows (256 / 512 / 1,024 patterns per call: the worker-group layout at ell = 1, 2 and the
    matrix-core encode at ell = 8), T and the estimate on sampled patterns and positions."""
    wl = BANDWIDTH
    O, order, holder, hpos = tables(wl)
    psi = gen.psi(wl, count=per_call)
    R = gen.shared_R(wl.m, ell)
    G = gen.given_G(wl, threads=THREADS)
    Gd = dev(G)
    pd = dev(psi)
    _, _, _, Bc = gcx.gc_decode_coeffs(pd, dev(order), dev(holder), dev(hpos), dev(R))
    T = gcx.gc_encode(Gd, pd, dev(order), Bc)
    ghat, sqerr = gcx.gc_reconstruct(T, dev(R), wl.d, psi=pd, gsum=gcx.gc_sum_chunks(Gd))
    L = -(-wl.d // ell)
    rng = np.random.default_rng(60 + ell)
    xs = sorted(set([0, 255, 256, 511, 512, 1023, 1024, L - 257, L - 1] + rng.choice(L, 40, replace=False).tolist()))
    pats = sorted(set([0, 1, per_call // 2, per_call - 1]))
    check_sampled(O, order, psi, R, G, "f32", T, ghat, pats, xs, ell)
    assert np.isfinite(host(sqerr)).all()
    del T, ghat, Bc, Gd
    torch.cuda.empty_cache()
