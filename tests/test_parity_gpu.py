"""GPU parity: every C-ABI call against the oracle on identical seeded inputs.

Stage by stage, each call receives inputs that come from the generators or
from the oracle (never from another GPU call) and is compared element by
element with the oracle:
  - coverage, decodability and coefficient error: bit-exact;
  - Bc: one fp32 rounding plus the fp64 solve's kappa^2 * 2^-53 error;
  - T and the estimate: the classical fp32 summation bound gamma_n * sum |terms|;
  - end to end: relative L2 error of the estimate <= 1e-5 at ell = 1 and, at
    ell >= 2, on every pattern whose matrices R[:, S_i] all have kappa_2 <= 100;
    the other ell >= 2 patterns are held to the cancellation-aware bound.
"""
from __future__ import annotations

import dataclasses
import functools

import numpy as np
import pytest

import oracle.assignment as OA
import oracle.protocol as OP
import oracle_runs as R_
from workloads import BANDWIDTH, HEADLINE, LARGE, SMALL, TINY, Workload, gen

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2405_19509_amd import gcx  # noqa: E402

U = R_.U

# ragged shapes: N > 64 lanes, d not a multiple of 4 / of ell, pattern counts not multiples of tiles
RAGGED = Workload(name="ragged_m70_d1001", N=70, m=70, s=5, d=1001, P=37, ells=(1, 3),
                  g_dtype="f32", pattern="uniform", forced_zero=7)
RAGGED_BF16 = dataclasses.replace(RAGGED, name="ragged_m70_d1000_bf16", d=1000, g_dtype="bf16")
LARGE_D16 = dataclasses.replace(LARGE, name="given_m200_d65536_bf16", d=1 << 16)
BANDWIDTH_D16 = dataclasses.replace(BANDWIDTH, name="given_m100_d65536", d=1 << 16)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


@functools.lru_cache(maxsize=None)
def tables(wl: Workload):
    O, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_CYCLIC, wl.N, wl.m, wl.s)
    assert (O == OA.cyclic_O(wl.N, wl.m, wl.s)).all()
    return O.astype(np.int64), order, holder, hpos


@functools.lru_cache(maxsize=None)
def patterns(wl: Workload, count: int, variant: str = "exact"):
    return gen.psi(wl, count=min(count, wl.P), variant=variant)


@functools.lru_cache(maxsize=None)
def given_G(wl: Workload):
    return gen.given_G(wl)


def G_torch(wl, G):
    if wl.g_dtype == "bf16":
        return dev(G.view(np.int16)).view(torch.bfloat16)
    return dev(G)


def run_decode(wl, psi, R):
    O, order, holder, hpos = tables(wl)
    cov, dec, cerr, Bc = gcx.gc_decode_coeffs(dev(psi), dev(order), dev(holder), dev(hpos), dev(R))
    return host(cov), host(dec), host(cerr), host(Bc)


def check_decode(wl, psi, R, per_worker=False):
    O, order, _, _ = tables(wl)
    ell = R.shape[0]
    cov, dec, cerr, Bc = run_decode(wl, psi, R)
    cov_ref = R_.coverage_all(O, psi)
    assert (cov == cov_ref).all()
    dec_ref = np.array([OP.decodable(O, p, ell) for p in psi])
    assert (dec == dec_ref.astype(np.uint8)).all()
    cerr_ref = np.array([OP.coef_err(O, p, ell) for p in psi])
    assert (cerr == cerr_ref).all()
    Bc_ref, kappa = R_.coefficients(O, psi, R, per_worker=per_worker)
    bound = R_.bc_bound(Bc_ref, kappa, O)
    diff = np.abs(Bc.astype(np.float64) - Bc_ref)
    worst = np.unravel_index(np.argmax(diff - bound), diff.shape)
    assert (diff <= bound).all(), f"Bc off at {worst}: {Bc[worst]} vs {Bc_ref[worst]} (bound {bound[worst]})"
    return Bc_ref, kappa


DECODE_CASES = [
    (TINY, 1, 100, True), (TINY, 2, 100, True), (TINY, 3, 100, True),
    (SMALL, 1, 1000, False), (SMALL, 2, 1000, False), (SMALL, 2, 60, True),
    (HEADLINE, 1, 400, False), (HEADLINE, 2, 400, False),
    (BANDWIDTH, 1, 60, False), (BANDWIDTH, 2, 60, False), (BANDWIDTH, 8, 60, False),
    (LARGE, 1, 12, False), (LARGE, 2, 12, False),
    (RAGGED, 1, 37, True), (RAGGED, 3, 37, False), (RAGGED, 7, 37, False),
]


@pytest.mark.parametrize("wl,ell,count,per_worker", DECODE_CASES,
                         ids=[f"{w.name}-l{e}-P{c}" for w, e, c, _ in DECODE_CASES])
def test_decode_parity(wl, ell, count, per_worker):
    psi = patterns(wl, count)
    R = gen.shared_R(wl.m, ell)
    check_decode(wl, psi, R, per_worker=per_worker)


@pytest.mark.parametrize("ell", [1, 2, 4])
def test_decode_parity_large_least_squares(ell):
    psi = patterns(LARGE, 12, "ls")
    assert (psi == 0).sum(axis=1).min() >= LARGE.ls_forced_zero
    check_decode(LARGE, psi, gen.shared_R(LARGE.m, ell))


@pytest.mark.parametrize("m", [200, 300])
def test_decode_cyclic_streamed_patterns(m):
    """The cyclic ell = 1 decode with more patterns than resident waves, so each wave walks
    several patterns (m = 200 and m = 300 workers: up to and past four psi entries per lane),
    and invalid patterns inside the walk: integers for every pattern, coefficients on sampled
    ones (the first, both sides of the first waves' second pattern, the invalid ones'
    neighbours, the last)."""
    wl = Workload(name=f"cyc_m{m}", N=m, m=m, s=9, d=64, P=20000, ells=(1,), pattern="uniform")
    O, order, holder, hpos = tables(wl)
    psi = patterns(wl, wl.P).copy()
    bad = [9000, 9001, 15555]
    psi[9000, 3] = wl.delta + 1
    psi[9001, m - 1] = -1
    psi[15555, 0] = wl.delta + 7
    R = gen.shared_R(m, 1)
    cov, dec, cerr, Bc = run_decode(wl, psi, R)
    ok = np.ones(wl.P, dtype=bool)
    ok[bad] = False
    assert (dec[bad] == gcx.GC_DEC_INVALID).all() and (Bc[bad] == 0).all()
    ref = np.zeros((wl.P, wl.N), dtype=np.int64)
    for t in range(wl.delta):
        ref += psi[:, (np.arange(wl.N) - t) % m] > t  # worker (i - t) mod N holds chunk i at position t
    assert (cov[ok] == ref[ok]).all()
    assert (dec[ok] == (ref[ok] >= 1).all(axis=1)).all()
    assert (cerr[ok] == np.maximum(0, 1 - ref[ok]).sum(axis=1)).all()
    rng = np.random.default_rng(37)
    sample = sorted(set([0, 1, 4095, 4096, 6143, 6144, 6145, 8191, 8192, 8999, 9002, 15554, 15556,
                         wl.P - 2, wl.P - 1] + rng.choice(wl.P, 9, replace=False).tolist()) - set(bad))
    Bc_ref, kappa = R_.coefficients(O, psi[sample], R)
    bound = R_.bc_bound(Bc_ref, kappa, O)
    diff = np.abs(Bc[sample].astype(np.float64) - Bc_ref)
    worst = np.unravel_index(np.argmax(diff - bound), diff.shape)
    assert (diff <= bound).all(), f"Bc off at pattern {sample[worst[0]]}, {worst[1:]}"


def test_decode_edge_patterns():
    """No worker done, all done, single worker done, s = 0, P not a multiple of 4."""
    wl = dataclasses.replace(TINY, name="tiny_edges")
    m, delta = wl.m, wl.delta
    psi = np.array([[0] * m, [delta] * m, [delta] + [0] * (m - 1), [1] * m, [delta - 1] * m],
                   dtype=np.int32)
    for ell in (1, 2, 3, 8):
        check_decode(wl, psi, gen.shared_R(m, ell), per_worker=True)
    wl0 = Workload(name="s0", N=9, m=9, s=0, d=16, P=3, ells=(1,), pattern="uniform")
    for ell in (1, 2):
        check_decode(wl0, patterns(wl0, 3), gen.shared_R(9, ell), per_worker=True)


def test_decode_invalid_psi():
    wl = TINY
    psi = patterns(wl, 10).copy()
    psi[3, 2] = wl.delta + 1
    psi[7, 0] = -1
    cov, dec, cerr, Bc = run_decode(wl, psi, gen.shared_R(wl.m, 2))
    assert dec[3] == gcx.GC_DEC_INVALID and dec[7] == gcx.GC_DEC_INVALID
    assert (Bc[3] == 0).all() and (Bc[7] == 0).all()
    ok = [p for p in range(10) if p not in (3, 7)]
    check_decode(wl, psi[ok], gen.shared_R(wl.m, 2))


def test_decode_explicit_order_sec2_2():
    """The non-cyclic example of Sec. 2.2 through GC_ASSIGN_ORDER: supports and coefficients."""
    import pins
    O = pins.sec2_2_O()
    _, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_ORDER, 5, 5, -1, O)
    R = gen.shared_R(5, 2)
    for psi_row, golden in (([5, 2, 0, 2, 3], "sec2_2_support_exact.txt"),
                            ([4, 2, 0, 2, 3], "sec2_2_support_approx.txt")):
        psi = np.array([psi_row], dtype=np.int32)
        cov, dec, cerr, Bc = gcx.gc_decode_coeffs(dev(psi), dev(order), dev(holder), dev(hpos), dev(R))
        cov, dec, cerr, Bc = host(cov), host(dec), host(cerr), host(Bc)
        assert (cov[0] == OP.coverage(O, psi[0])).all()
        assert cerr[0] == OP.coef_err(O, psi[0], 2)
        B_ref = OP.encoding_matrix(O, psi[0], R)
        Bc_ref = OP.compact(B_ref, O, 2)
        assert np.allclose(Bc[0], Bc_ref, rtol=4 * U, atol=1e-6)
        # the support of B rebuilt from Bc is the printed one
        supp = np.zeros((5, 10), dtype=bool)
        for j in range(5):
            for t in range(order.shape[1]):
                i = order[j, t]
                if i >= 0:
                    supp[j, 2 * i:2 * i + 2] = Bc[0, j, t] != 0
        assert (supp == np.array(pins.load_rows(golden), dtype=bool)).all()


# ---------------------------------------------------------------------------
# encode and combine, stage by stage on oracle-made inputs
# ---------------------------------------------------------------------------

ENC_CASES = [
    (TINY, 1, 100), (TINY, 2, 100), (TINY, 3, 100),
    (SMALL, 1, 40), (SMALL, 2, 40),
    (HEADLINE, 1, 12), (HEADLINE, 2, 12),
    (BANDWIDTH_D16, 1, 6), (BANDWIDTH_D16, 2, 6), (BANDWIDTH_D16, 8, 6),
    (LARGE_D16, 1, 3), (LARGE_D16, 2, 3),
    (RAGGED, 1, 37), (RAGGED, 3, 37), (RAGGED_BF16, 3, 37),
]


def _data_G(wl):
    if wl.n is not None:
        X, y, w = gen.regression_data(wl)
        return R_.chunk_grads(X, y, w, wl.loss).astype(np.float32)
    return given_G(wl)


@pytest.mark.parametrize("wl,ell,count", ENC_CASES, ids=[f"{w.name}-l{e}-P{c}" for w, e, c in ENC_CASES])
def test_encode_and_reconstruct_parity(wl, ell, count):
    O, order, holder, hpos = tables(wl)
    psi = patterns(wl, count)
    R = gen.shared_R(wl.m, ell)
    Bc_ref, _ = R_.coefficients(O, psi, R)
    Bc32 = Bc_ref.astype(np.float32)
    G = _data_G(wl)
    Gw = OP.widen(G, wl.g_dtype)
    # encode on identical inputs: G, psi and the oracle's coefficients rounded to fp32
    # T starts as NaN: rows of workers that transmit nothing (psi = 0) must stay untouched
    Td = torch.full((len(psi), wl.m, -(-wl.d // ell)), float("nan"), device="cuda")
    T = host(gcx.gc_encode(G_torch(wl, G), dev(psi), dev(order), dev(Bc32), T=Td))
    T_ref, M, nterm = R_.encode_ref(Bc32.astype(np.float64), psi, order, Gw, ell)
    sent = psi > 0
    assert np.isnan(T[~sent]).all()
    bound = R_.encode_bound(nterm, M, wl.g_dtype)
    diff = np.abs(T[sent].astype(np.float64) - T_ref[sent])
    assert (diff <= bound[sent]).all(), f"T off by {np.max(diff - bound[sent])}"
    # combine on identical inputs: the oracle's T rounded to fp32
    T32 = T_ref.astype(np.float32)
    gsum_ref = Gw.sum(axis=0)
    gsum32 = gsum_ref.astype(np.float32)
    # the rows of non-transmitting workers are poisoned: given psi, they must not be read
    T32_poison = T32.copy()
    T32_poison[~sent] = np.nan
    ghat, sqerr = gcx.gc_reconstruct(dev(T32_poison), dev(R), wl.d, psi=dev(psi), gsum=dev(gsum32))
    ghat, sqerr = host(ghat), host(sqerr)
    gh_ref, mag = R_.reconstruct_ref(T32.astype(np.float64), R, wl.d)
    gb = R_.gamma(wl.m) * mag
    gdiff = np.abs(ghat.astype(np.float64) - gh_ref)
    assert (gdiff <= gb).all(), f"ghat off by {np.max(gdiff - gb)}"
    se_ref = ((gh_ref - gsum32.astype(np.float64)) ** 2).sum(axis=1)
    E = np.sqrt((gb ** 2).sum(axis=1))
    assert (np.abs(sqerr - se_ref) <= 2 * np.sqrt(se_ref) * E + E * E + 1e-12 * se_ref).all()
    # error-only mode gives the same sqerr
    _, sq2 = gcx.gc_reconstruct(dev(T32_poison), dev(R), wl.d, psi=dev(psi), gsum=dev(gsum32),
                                want_ghat=False)
    assert (host(sq2) == sqerr).all()


def test_encode_and_reconstruct_edge_patterns():
    """No worker done (nothing transmitted: the estimate is 0 and the squared error |gsum|^2),
    all done, a single worker done, one chunk each, all but the last chunk; the combine takes
    several items per block at ell = 1 and 2 (one with no transmitting row) and one at ell = 8."""
    wl = dataclasses.replace(TINY, name="tiny_edges_ec")
    m, delta = wl.m, wl.delta
    psi = np.array([[0] * m, [delta] * m, [delta] + [0] * (m - 1), [1] * m, [delta - 1] * m],
                   dtype=np.int32)
    O, order, _, _ = tables(wl)
    G = _data_G(wl)
    Gw = OP.widen(G, wl.g_dtype)
    gsum32 = Gw.sum(axis=0).astype(np.float32)
    sent = psi > 0
    for ell in (1, 2, 8):
        R = gen.shared_R(m, ell)
        Bc32 = R_.coefficients(O, psi, R)[0].astype(np.float32)
        Td = torch.full((len(psi), m, -(-wl.d // ell)), float("nan"), device="cuda")
        T = host(gcx.gc_encode(G_torch(wl, G), dev(psi), dev(order), dev(Bc32), T=Td))
        T_ref, M, nterm = R_.encode_ref(Bc32.astype(np.float64), psi, order, Gw, ell)
        assert np.isnan(T[~sent]).all()
        bound = R_.encode_bound(nterm, M, wl.g_dtype)[sent]
        assert (np.abs(T[sent].astype(np.float64) - T_ref[sent]) <= bound).all()
        T32 = T_ref.astype(np.float32)  # rows of workers with psi = 0 are zero in the oracle's T
        T32_poison = T32.copy()
        T32_poison[~sent] = np.nan
        ghat, sq = gcx.gc_reconstruct(dev(T32_poison), dev(R), wl.d, psi=dev(psi), gsum=dev(gsum32))
        ghat, sq = host(ghat), host(sq)
        assert (ghat[0] == 0).all()
        assert sq[0] == pytest.approx(float((gsum32.astype(np.float64) ** 2).sum()), rel=1e-12)
        gh_ref, mag = R_.reconstruct_ref(T32.astype(np.float64), R, wl.d)
        assert (np.abs(ghat.astype(np.float64) - gh_ref) <= R_.gamma(m) * mag).all()
        se_ref = ((gh_ref - gsum32.astype(np.float64)) ** 2).sum(axis=1)
        E = np.sqrt(((R_.gamma(m) * mag) ** 2).sum(axis=1))
        assert (np.abs(sq - se_ref) <= 2 * np.sqrt(se_ref) * E + E * E + 1e-12 * se_ref).all()


# worker-group encode layout: many chunks per slice, so the all-chunk layout does not fit;
# odd L (one float per lane), padding (ell does not divide d), bf16, 1 to 7 patterns per call
GROUP_CASES = [
    (Workload(name="group_m130_d3002", N=130, m=130, s=3, d=3002, P=7, ells=(3,), pattern="uniform"), 3, 1),
    (Workload(name="group_m130_d3002", N=130, m=130, s=3, d=3002, P=7, ells=(3,), pattern="uniform"), 3, 7),
    (Workload(name="group_m200_d4001_bf16", N=200, m=200, s=5, d=4001, P=3, ells=(4,), g_dtype="bf16",
              pattern="uniform"), 4, 3),
    (Workload(name="group_m120_d8192", N=120, m=120, s=9, d=8192, P=5, ells=(2,), pattern="uniform"), 2, 5),
]


@pytest.mark.parametrize("wl,ell,count", GROUP_CASES, ids=[f"{w.name}-l{e}-P{c}" for w, e, c in GROUP_CASES])
def test_encode_worker_groups(wl, ell, count):
    O, order, _, _ = tables(wl)
    psi = patterns(wl, count)
    R = gen.shared_R(wl.m, ell)
    Bc32 = R_.coefficients(O, psi, R)[0].astype(np.float32)
    G = given_G(wl)
    # rows of workers with psi = 0 transmit nothing and must stay untouched
    Td = torch.full((len(psi), wl.m, -(-wl.d // ell)), float("nan"), device="cuda")
    T = host(gcx.gc_encode(G_torch(wl, G), dev(psi), dev(order), dev(Bc32), T=Td))
    T_ref, M, nterm = R_.encode_ref(Bc32.astype(np.float64), psi, order, OP.widen(G, wl.g_dtype), ell)
    sent = psi > 0
    assert np.isnan(T[~sent]).all()
    bound = R_.encode_bound(nterm, M, wl.g_dtype)[sent]
    assert (np.abs(T[sent].astype(np.float64) - T_ref[sent]) <= bound).all()


# matrix-core encode: at least one full 32-pattern tile and delta*ell >= 32 terms per output
MF_CASES = [
    (Workload(name="mf_m100_d4096", N=100, m=100, s=9, d=4096, P=40, ells=(8,), pattern="uniform"), 8, 40),
    # fp32 on the bf16 matrix cores: two full 64-pattern windows and one of 2, odd L
    (Workload(name="mf_m100_d2052", N=100, m=100, s=9, d=2052, P=130, ells=(8,), pattern="uniform"), 8, 130),
    (Workload(name="mf_m200_d2001_bf16", N=200, m=200, s=7, d=2001, P=33, ells=(4,), g_dtype="bf16",
              pattern="uniform"), 4, 33),
]


@pytest.mark.parametrize("wl,ell,count", MF_CASES, ids=[f"{w.name}-l{e}-P{c}" for w, e, c in MF_CASES])
def test_encode_matrix_cores(wl, ell, count):
    """32-pattern tiles on the matrix cores: a partial last tile, odd L (bf16), padding."""
    O, order, _, _ = tables(wl)
    psi = patterns(wl, count)
    R = gen.shared_R(wl.m, ell)
    Bc32 = R_.coefficients(O, psi, R)[0].astype(np.float32)
    G = given_G(wl)
    Td = torch.full((len(psi), wl.m, -(-wl.d // ell)), float("nan"), device="cuda")
    T = host(gcx.gc_encode(G_torch(wl, G), dev(psi), dev(order), dev(Bc32), T=Td))
    T_ref, M, nterm = R_.encode_ref(Bc32.astype(np.float64), psi, order, OP.widen(G, wl.g_dtype), ell)
    sent = psi > 0
    assert np.isnan(T[~sent]).all()
    bound = R_.encode_bound(nterm, M, wl.g_dtype)[sent]
    assert (np.abs(T[sent].astype(np.float64) - T_ref[sent]) <= bound).all()


# matrix-core encode with (pattern, worker) rows: fewer than 32 patterns per call, >= 32 terms
MR_WL = Workload(name="mr_m100_d4099", N=100, m=100, s=15, d=4099, P=16, ells=(2,), pattern="uniform")
MR_WL_BF16 = Workload(name="mr_m200_d4001_bf16", N=200, m=200, s=19, d=4001, P=3, ells=(4,),
                      g_dtype="bf16", pattern="uniform")
MR_CASES = [(MR_WL, 2, 1), (MR_WL, 2, 2), (MR_WL, 2, 7), (MR_WL, 2, 16), (MR_WL_BF16, 4, 3)]


def _encode_against_oracle(O, order, psi, R, G, g_dtype, ell, d, shift=0):
    """The encode of G (placed `shift` elements past an aligned device allocation) against
    the oracle's, on the oracle's coefficients rounded to fp32."""
    Bc32 = R_.coefficients(O, psi, R)[0].astype(np.float32)
    Gt = dev(G.view(np.int16)).view(torch.bfloat16) if g_dtype == "bf16" else dev(G)
    if shift:
        buf = torch.empty(Gt.numel() + shift, dtype=Gt.dtype, device="cuda")
        moved = buf[shift:].view(Gt.shape)
        moved.copy_(Gt)
        Gt = moved
    Td = torch.full((len(psi), O.shape[1], -(-d // ell)), float("nan"), device="cuda")
    T = host(gcx.gc_encode(Gt, dev(psi), dev(order), dev(Bc32), T=Td))
    T_ref, M, nterm = R_.encode_ref(Bc32.astype(np.float64), psi, order, OP.widen(G, g_dtype), ell)
    sent = psi > 0
    assert np.isnan(T[~sent]).all()
    bound = R_.encode_bound(nterm, M, g_dtype)[sent]
    assert (np.abs(T[sent].astype(np.float64) - T_ref[sent]) <= bound).all()


@pytest.mark.parametrize("ell", [1, 2])
@pytest.mark.parametrize("g_dtype,shift", [("f32", 0), ("f32", 1), ("bf16", 0), ("bf16", 1)])
def test_encode_all_chunk_staging(g_dtype, shift, ell):
    """The all-chunk layout with its slices staged straight into LDS 16 bytes at a time (G
    16-byte aligned, d and L whole 16-byte pieces), and element by element when G sits one
    element off that alignment; 23 x 40 = 920 rows: two 256-row metadata groups in the first
    block, a ragged second block."""
    wl = Workload(name=f"allchunk_m40_d4096_{g_dtype}", N=40, m=40, s=3, d=4096, P=23, ells=(ell,),
                  g_dtype=g_dtype, pattern="uniform")
    O, order, _, _ = tables(wl)
    _encode_against_oracle(O, order, patterns(wl, 23), gen.shared_R(wl.m, ell), given_G(wl), g_dtype,
                           ell, wl.d, shift=shift)


@pytest.mark.parametrize("wl,ell,count", MR_CASES, ids=[f"{w.name}-l{e}-P{c}" for w, e, c in MR_CASES])
def test_encode_matrix_rows(wl, ell, count):
    """16 rows of (pattern, worker) per tile on the matrix cores: 1 to 16 patterns per call,
    odd L, padding, bf16."""
    O, order, _, _ = tables(wl)
    _encode_against_oracle(O, order, patterns(wl, count), gen.shared_R(wl.m, ell), given_G(wl),
                           wl.g_dtype, ell, wl.d)


def test_encode_matrix_rows_spilled_union():
    """A random 16-regular support (Algorithm 2 ordering): the chunks of 8 workers no longer fit
    the matrix-rows layout's slots, so its blocks take the vector path."""
    import oracle.ordering as OO
    m, nu, ell, d = 100, 16, 2, 4099
    A = gen.random_regular_graph(m, nu)
    O = OO.chunk_ordering(A)
    _, order, _, _ = gcx.gc_assign(gcx.GC_ASSIGN_ORDER, m, m, -1, O.astype(np.int32), nu, nu)
    g = np.random.default_rng(41)
    psi = g.integers(0, nu + 1, size=(2, m)).astype(np.int32)
    G = g.standard_normal((m, d)).astype(np.float32)
    _encode_against_oracle(O.astype(np.int64), order, psi, gen.shared_R(m, ell), G, "f32", ell, d)


# bf16 chunk gradients past the all-chunk layout: the bf16 matrix cores, 32 rows of (pattern,
# worker) per tile, coefficients split in three bf16 parts
MX_WL = Workload(name="mx_m200_d4000_bf16", N=200, m=200, s=19, d=4000, P=40, ells=(1, 2, 4),
                 g_dtype="bf16", pattern="uniform", forced_zero=30)
MX_CASES = [
    (MX_WL, 1, 1), (MX_WL, 1, 3), (MX_WL, 1, 8), (MX_WL, 2, 16), (MX_WL, 4, 33), (MX_WL, 4, 130),
    (dataclasses.replace(MX_WL, name="mx_m70_d4001_bf16", N=70, m=70, s=9, d=4001), 3, 8),   # ragged, 70 % 4
    (dataclasses.replace(MX_WL, name="mx_m100_d81920_bf16", N=100, m=100, s=9, d=2048 * 40), 2, 5),
    (dataclasses.replace(MX_WL, name="mx_m200_d1024_bf16", d=1024), 8, 4),    # too many rows: other path
]


@pytest.mark.parametrize("wl,ell,count", MX_CASES, ids=[f"{w.name}-l{e}-P{c}" for w, e, c in MX_CASES])
def test_encode_bf16_matrix_cores(wl, ell, count):
    """bf16 gradients on the bf16 matrix cores: 1 to 33 patterns per call (32 / 8 / 4 / 2 / 1
    workers per tile, two pattern tiles), 128-candidate windows (ell = 2 to 4; 130 patterns:
    a full window of 128 patterns and one of 2), ragged d and ell not dividing d
    (element-wise staging), a group count that does not divide m, straggler rows untouched;
    and a shape whose staged rows do not fit (ell = 8), which takes the worker-group path."""
    O, order, _, _ = tables(wl)
    _encode_against_oracle(O, order, patterns(wl, count), gen.shared_R(wl.m, ell), given_G(wl), "bf16",
                           ell, wl.d)


def test_encode_bf16_matrix_cores_misaligned_and_spilled_union():
    """G one element off 16-byte alignment (element-wise staging); and a random 16-regular
    support ordered by Algorithm 2, whose worker groups use more chunks than their slots,
    so each block walks its workers one at a time (64- and 128-candidate windows)."""
    import oracle.ordering as OO
    wl = dataclasses.replace(MX_WL, name="mx_shift_m200_d4096_bf16", d=4096)
    O, order, _, _ = tables(wl)
    _encode_against_oracle(O, order, patterns(wl, 4), gen.shared_R(wl.m, 2), given_G(wl), "bf16", 2, wl.d,
                           shift=1)
    m, nu, d = 100, 16, 3000
    A = gen.random_regular_graph(m, nu)
    O2 = OO.chunk_ordering(A)
    _, order2, _, _ = gcx.gc_assign(gcx.GC_ASSIGN_ORDER, m, m, -1, O2.astype(np.int32), nu, nu)
    g = np.random.default_rng(43)
    psi = g.integers(0, nu + 1, size=(4, m)).astype(np.int32)
    G = gen.f32_to_bf16_bits(g.standard_normal((m, d)).astype(np.float32))
    _encode_against_oracle(O2.astype(np.int64), order2, psi, gen.shared_R(m, 1), G, "bf16", 1, d)
    # ell = 2: 128-candidate windows (4 patterns x 32 workers), whose unions spill too
    _encode_against_oracle(O2.astype(np.int64), order2, psi, gen.shared_R(m, 2), G, "bf16", 2, d)


@pytest.mark.parametrize("wl,ell", [(TINY, 2), (GROUP_CASES[3][0], 2)], ids=["all-chunk", "worker-group"])
def test_encode_clamps_psi(wl, ell):
    """psi outside [0, delta] is clamped, in both encode layouts: a negative count sends
    nothing, a count past the load encodes the whole order."""
    O, order, _, _ = tables(wl)
    g = np.random.default_rng(31)
    P = 6
    psi = g.integers(-3, wl.delta + 4, size=(P, wl.m)).astype(np.int32)
    Bc = g.standard_normal((P, wl.m, wl.delta, ell)).astype(np.float32)
    G = given_G(wl)
    Td = torch.full((P, wl.m, -(-wl.d // ell)), float("nan"), device="cuda")
    T = host(gcx.gc_encode(G_torch(wl, G), dev(psi), dev(order), dev(Bc), T=Td))
    clamped = np.clip(psi, 0, wl.delta)
    T_ref, M, nterm = R_.encode_ref(Bc.astype(np.float64), clamped, order, OP.widen(G, wl.g_dtype), ell)
    sent = clamped > 0
    assert np.isnan(T[~sent]).all()
    assert (np.abs(T[sent].astype(np.float64) - T_ref[sent]) <= R_.encode_bound(nterm, M, wl.g_dtype)[sent]).all()


@pytest.mark.parametrize("ell,d", [(1, 512), (2, 513)])
def test_encode_many_chunks(ell, d):
    """5,000 chunks, 8 workers each holding 6 (one worker 4) of them in an explicit order:
    more chunks than the per-group chunk map holds, so single-worker groups; random
    coefficients (the encode is linear in them) against the oracle's encode."""
    N, m, delta, P = 5000, 8, 6, 5
    g = np.random.default_rng(21 + ell)
    order = np.stack([g.choice(N, size=delta, replace=False) for _ in range(m)]).astype(np.int32)
    order[3, 4:] = -1                                    # a worker with a shorter order
    psi = g.integers(0, delta + 1, size=(P, m)).astype(np.int32)
    psi[:, 3] = np.minimum(psi[:, 3], 4)
    Bc = g.standard_normal((P, m, delta, ell)).astype(np.float32)
    G = g.standard_normal((N, d)).astype(np.float32)
    T = host(gcx.gc_encode(dev(G), dev(psi), dev(order), dev(Bc)))
    T_ref, M, nterm = R_.encode_ref(Bc.astype(np.float64), psi, order, G.astype(np.float64), ell)
    sent = psi > 0
    assert (np.abs(T[sent].astype(np.float64) - T_ref[sent]) <= R_.encode_bound(nterm, M, "f32")[sent]).all()


def _uneven_assignment(seed=5):
    """9 chunks over 6 workers, 2 or 3 holders per chunk, loads 3 to 5, orders shuffled."""
    N, m = 9, 6
    g = np.random.default_rng(seed)
    S = np.zeros((N, m), dtype=bool)
    for i in range(N):
        S[i, [i % m, (i + 2) % m]] = True
        if i % 3 == 0:
            S[i, (i + 3) % m] = True
    O = np.zeros((N, m), dtype=np.int32)
    for j in range(m):
        rows = np.flatnonzero(S[:, j])
        O[rows, j] = g.permutation(len(rows)) + 1
    return O


@pytest.mark.parametrize("ell", [1, 2])
def test_uneven_non_square_assignment(ell):
    """N != m with unequal loads and replications, through GC_ASSIGN_ORDER: coefficients,
    encode, combine and the PS-side estimate against the oracle on every valid psi drawn."""
    O = _uneven_assignment()
    N, m = O.shape
    _, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_ORDER, N, m, -1, O)
    loads = (O != 0).sum(axis=0)
    g = np.random.default_rng(11 + ell)
    # 40 patterns uniform over each worker's progress, 20 with every worker at most one short
    psi = np.concatenate([np.stack([g.integers(0, loads + 1) for _ in range(40)]),
                          np.maximum(loads - g.integers(0, 2, size=(20, m)), 0)]).astype(np.int32)
    R = gen.shared_R(m, ell)
    d = 301
    G = g.standard_normal((N, d)).astype(np.float32)
    cov, dec, cerr, Bc = gcx.gc_decode_coeffs(dev(psi), dev(order), dev(holder), dev(hpos), dev(R))
    cov, dec, cerr = host(cov), host(dec), host(cerr)
    for p in range(len(psi)):
        c = OP.coverage(O, psi[p])
        assert (cov[p] == c).all() and dec[p] == int((c >= ell).all())
        assert cerr[p] == OP.coef_err(O, psi[p], ell)
    Bc_ref, kappa = R_.coefficients(O, psi, R)
    assert (np.abs(host(Bc).astype(np.float64) - Bc_ref) <= R_.bc_bound(Bc_ref, kappa, O)).all()
    # encode + combine on the oracle's coefficients
    Bc32 = Bc_ref.astype(np.float32)
    T = host(gcx.gc_encode(dev(G), dev(psi), dev(order), dev(Bc32)))
    T_ref, M, nterm = R_.encode_ref(Bc32.astype(np.float64), psi, order, G.astype(np.float64), ell)
    sent = psi > 0
    assert (np.abs(T[sent] - T_ref[sent]) <= R_.encode_bound(nterm, M, "f32")[sent]).all()
    T32 = T_ref.astype(np.float32)
    gh, _ = gcx.gc_reconstruct(dev(T32), dev(R), d, psi=dev(psi))
    gh_ref, mag = R_.reconstruct_ref(T32.astype(np.float64), R, d)
    assert (np.abs(host(gh) - gh_ref) <= R_.gamma(m) * mag).all()
    # the PS-side estimate from the chunk gradients
    G64 = G.astype(np.float64)
    gsum = G64.sum(axis=0).astype(np.float32)
    ghd, sq = gcx.gc_decode_direct(dev(G), dev(psi), dev(order), dev(holder), dev(hpos), dev(R),
                                   gsum=dev(gsum))
    ghd, sq = host(ghd).astype(np.float64), host(sq)
    ref, mg, kap = R_.direct_ref(O, psi, R, G64)
    magG = np.tile(np.abs(R_.gblocks(G64, ell)).sum(axis=(0, 1)), ell)[:d]
    bound = 2 * R_.gamma(N * ell + 2) * mg + 1e-13 * (kap ** 2)[:, None] * magG
    assert (np.abs(ghd - ref) <= bound + 1e-30).all()
    # sqerr against the GPU's own estimate (fp32 differences, fp64 sum)
    se = ((ghd - gsum.astype(np.float64)) ** 2).sum(axis=1)
    assert np.allclose(sq, se, rtol=1e-5, atol=1e-9)
    assert (dec == (np.abs(ghd - gsum).max(axis=1) <= 1e-3 * np.abs(gsum).max())).all()


def test_sum_chunks():
    for wl in (TINY, RAGGED, RAGGED_BF16, LARGE_D16):
        G = _data_G(wl)
        Gw = OP.widen(G, wl.g_dtype)
        gs = host(gcx.gc_sum_chunks(G_torch(wl, G))).astype(np.float64)
        want = Gw.sum(axis=0)
        assert (np.abs(gs - want) <= 2 * U * np.abs(want) + 1e-30).all()


# ---------------------------------------------------------------------------
# chunk gradients
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("wl", [TINY, SMALL, HEADLINE], ids=lambda w: w.name)
def test_chunk_grads_parity(wl):
    X, y, w = gen.regression_data(wl)
    G = host(gcx.gc_chunk_grads(dev(X), dev(y), dev(w), 0 if wl.loss == "linear" else 1))
    G_ref = R_.chunk_grads(X, y, w, wl.loss)
    rel = np.linalg.norm(G - G_ref, axis=1) / np.linalg.norm(G_ref, axis=1)
    assert rel.max() <= 1e-5, rel.max()


def test_chunk_grads_multi_point_and_ragged():
    wl = Workload(name="ragged_reg", N=5, m=5, s=1, d=1001, P=1, ells=(1,), n=37, loss="logistic",
                  x_std=0.05, w_std=0.1)
    X, y, _ = gen.regression_data(wl)
    W = gen.eval_points(wl, 3)
    G = host(gcx.gc_chunk_grads(dev(X), dev(y), dev(W), gcx.GC_LOSS_LOGISTIC))
    G_ref = R_.chunk_grads(X, y, W, "logistic")
    rel = np.linalg.norm(G - G_ref, axis=-1) / np.linalg.norm(G_ref, axis=-1)
    assert G.shape == (3, 5, 1001) and rel.max() <= 1e-5


MFMA_CASES = [(TINY, 16), (SMALL, 64), (HEADLINE, 32)]


@pytest.mark.parametrize("wl,b", MFMA_CASES, ids=[f"{w.name}-b{b}" for w, b in MFMA_CASES])
def test_chunk_grads_many_points_mfma(wl, b):
    """b >= 16 points: the two contractions run on the fp32 matrix cores."""
    X, y, _ = gen.regression_data(wl)
    W = gen.eval_points(wl, b)
    G = host(gcx.gc_chunk_grads(dev(X), dev(y), dev(W), 0 if wl.loss == "linear" else 1))
    G_ref = R_.chunk_grads(X, y, W, wl.loss)
    rel = np.linalg.norm(G - G_ref, axis=-1) / np.linalg.norm(G_ref, axis=-1)
    assert G.shape == (b, wl.N, wl.d) and rel.max() <= 1e-5, rel.max()


def test_chunk_grads_mfma_ragged_tiles():
    """Row, point and column counts that are not multiples of the 128 x 128 tiles; with 7
    chunks of d = 9000, more output tiles than resident blocks, so each block of G = U^T X
    walks several tiles (ragged ones among them) as one stream of stages."""
    for N, d, bs in ((3, 1000, (20, 132)), (7, 9000, (132, 256))):
        wl = Workload(name=f"ragged_mfma_N{N}_d{d}", N=N, m=N, s=1, d=d, P=1, ells=(1,), n=37,
                      loss="logistic", x_std=0.05, w_std=0.1)
        X, y, _ = gen.regression_data(wl)
        for b in bs:
            W = gen.eval_points(wl, b)
            G = host(gcx.gc_chunk_grads(dev(X), dev(y), dev(W), gcx.GC_LOSS_LOGISTIC))
            G_ref = R_.chunk_grads(X, y, W, "logistic")
            rel = np.linalg.norm(G - G_ref, axis=-1) / np.linalg.norm(G_ref, axis=-1)
            assert rel.max() <= 1e-5, (N, d, b, rel.max())


# ---------------------------------------------------------------------------
# end to end: GPU pipeline vs full oracle
# ---------------------------------------------------------------------------

E2E_CASES = [(TINY, 1, 100), (TINY, 2, 100), (TINY, 3, 100), (SMALL, 1, 100), (SMALL, 2, 100),
             (HEADLINE, 1, 40), (HEADLINE, 2, 40), (RAGGED, 1, 37), (RAGGED, 3, 37)]


@pytest.mark.parametrize("wl,ell,count", E2E_CASES, ids=[f"{w.name}-l{e}-P{c}" for w, e, c in E2E_CASES])
def test_end_to_end(wl, ell, count):
    O, order, holder, hpos = tables(wl)
    psi = patterns(wl, count)
    R = gen.shared_R(wl.m, ell)
    if wl.n is not None:
        X, y, w = gen.regression_data(wl)
        Gd = gcx.gc_chunk_grads(dev(X), dev(y), dev(w), 0 if wl.loss == "linear" else 1)
        G_ref = R_.chunk_grads(X, y, w, wl.loss)
    else:
        G = given_G(wl)
        Gd = G_torch(wl, G)
        G_ref = OP.widen(G, wl.g_dtype)
    gsum = gcx.gc_sum_chunks(Gd)
    _, _, _, Bc = gcx.gc_decode_coeffs(dev(psi), dev(order), dev(holder), dev(hpos), dev(R))
    T = gcx.gc_encode(Gd, dev(psi), dev(order), Bc)
    ghat, sqerr = gcx.gc_reconstruct(T, dev(R), wl.d, psi=dev(psi), gsum=gsum)
    ghat, sqerr = host(ghat).astype(np.float64), host(sqerr)
    gh_ref = R_.end_to_end(O, psi, R, G_ref)
    rel = np.linalg.norm(ghat - gh_ref, axis=1) / np.maximum(np.linalg.norm(gh_ref, axis=1), 1e-300)
    if ell == 1:
        assert rel.max() <= 1e-5, rel.max()
    else:
        # cancellation-aware bound: the combine's inputs are as large as sum_j |R||T_j|
        Bc_ref, kappa = R_.coefficients(O, psi, R)
        T_ref, M, nterm = R_.encode_ref(Bc_ref, psi, order, G_ref, ell)
        _, mag = R_.reconstruct_ref(np.abs(T_ref) + M, R, wl.d)
        allowed = np.maximum(1e-5, 4 * R_.gamma(wl.m + ell * wl.delta + 2) *
                             np.linalg.norm(mag, axis=1) / np.maximum(np.linalg.norm(gh_ref, axis=1), 1e-300))
        assert (rel <= allowed).all(), (rel / allowed).max()
        # patterns whose every R[:, S_i] has kappa_2 <= 100 are held to the plain 1e-5
        well = kappa.max(axis=1) <= 100
        assert well.sum() >= len(psi) // 3, well.sum()
        print(f"ell={ell}: rel-L2 max {rel[well].max():.2e} over {well.sum()} patterns with kappa <= 100")
        assert rel[well].max() <= 1e-5, rel[well].max()
        if (~well).any():
            kmax = kappa.max(axis=1)[~well]
            print(f"ell={ell}: other patterns: max rel / (8 kappa_max u) = {(rel[~well] / (8 * kmax * U)).max():.2e}")
    se_ref = ((ghat - G_ref.sum(axis=0)) ** 2).sum(axis=1)
    assert np.allclose(sqerr, se_ref, rtol=1e-4, atol=1e-10 * float((G_ref.sum(axis=0) ** 2).sum()))
