"""GPU parity at the ABI's limits: m = N = GC_MAX_M = 1024 workers, delta = GC_MAX_DELTA = 64,
ell = GC_MAX_ELL = 8, a ragged d.  The tables no longer fit the two-phase decode's LDS (the
one-phase kernel runs), the encode's chunk slices spill past the worker-group LDS capacity
(the L2 path), the combine compacts 1,024 rows, and the PS-side estimate runs its k-staged
kernel (K = N ell = 8,192).  Everything against the oracle on the same inputs."""
from __future__ import annotations

import numpy as np
import pytest

import oracle.assignment as OA
import oracle.protocol as OP
import oracle_runs as R_
from workloads import gen

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2405_19509_amd import gcx  # noqa: E402


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def test_abi_limits():
    m, s, ell, d = gcx.GC_MAX_M, gcx.GC_MAX_DELTA - 1, gcx.GC_MAX_ELL, 1027
    delta = s + 1
    O, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_CYCLIC, m, m, s)
    assert (O == OA.cyclic_O(m, m, s)).all()
    O = O.astype(np.int64)
    g = np.random.default_rng(1024)
    # one pattern with little progress (coverage 0..12 < ell for many chunks: least squares),
    # one where every worker is done (decodable)
    psi = np.stack([g.integers(0, 13, size=m), np.full(m, delta)]).astype(np.int32)
    R = gen.shared_R(m, ell)
    cov, dec, cerr, Bc = gcx.gc_decode_coeffs(dev(psi), dev(order), dev(holder), dev(hpos), dev(R))
    cov, dec, cerr, Bc = host(cov), host(dec), host(cerr), host(Bc)
    for p in range(len(psi)):
        c = OP.coverage(O, psi[p])
        assert (cov[p] == c).all()
        assert dec[p] == int((c >= ell).all()) and cerr[p] == OP.coef_err(O, psi[p], ell)
    assert dec[0] == gcx.GC_DEC_NO and dec[1] == gcx.GC_DEC_YES
    Bc_ref, kappa = R_.coefficients(O, psi, R)
    assert (np.abs(Bc.astype(np.float64) - Bc_ref) <= R_.bc_bound(Bc_ref, kappa, O)).all()

    # encode on the oracle's coefficients; straggler rows stay untouched
    G = g.standard_normal((m, d)).astype(np.float32)
    Bc32 = Bc_ref.astype(np.float32)
    L = -(-d // ell)
    Td = torch.full((len(psi), m, L), float("nan"), device="cuda")
    T = host(gcx.gc_encode(dev(G), dev(psi), dev(order), dev(Bc32), T=Td))
    T_ref, M, nterm = R_.encode_ref(Bc32.astype(np.float64), psi, order, G.astype(np.float64), ell)
    sent = psi > 0
    assert np.isnan(T[~sent]).all()
    assert (np.abs(T[sent].astype(np.float64) - T_ref[sent]) <= R_.encode_bound(nterm, M, "f32")[sent]).all()

    # combine on the oracle's transmitted vectors
    T32 = T_ref.astype(np.float32)
    gh, _ = gcx.gc_reconstruct(dev(T32), dev(R), d, psi=dev(psi))
    gh_ref, mag = R_.reconstruct_ref(T32.astype(np.float64), R, d)
    assert (np.abs(host(gh).astype(np.float64) - gh_ref) <= R_.gamma(m) * mag).all()

    # the PS-side estimate from the chunk gradients
    G64 = G.astype(np.float64)
    ghd, _ = gcx.gc_decode_direct(dev(G), dev(psi), dev(order), dev(holder), dev(hpos), dev(R))
    ref, mg, kap = R_.direct_ref(O, psi, R, G64)
    magG = np.tile(np.abs(R_.gblocks(G64, ell)).sum(axis=(0, 1)), ell)[:d]
    bound = 2 * R_.gamma(m * ell + 2) * mg + 1e-13 * (kap ** 2)[:, None] * magG
    assert (np.abs(host(ghd).astype(np.float64) - ref) <= bound + 1e-30).all()
    # the decodable pattern recovers the sum of the chunk gradients
    assert np.abs(host(ghd)[1] - G64.sum(axis=0)).max() <= 1e-3 * np.abs(G64).sum(axis=0).max()
