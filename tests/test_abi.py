"""The C-ABI library on the CPU: it loads, exports every declared symbol, and its
host-only entry points and host-side validation behave as documented."""
import os
import re

import numpy as np
import pytest

import oracle.assignment as OA
from paper_2405_19509_amd import gcx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gcx.h")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gc_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_hot_path():
    syms = declared_symbols()
    for name in ("gc_assign", "gc_chunk_grads", "gc_encode", "gc_decode_coeffs", "gc_reconstruct"):
        assert name in syms


def test_library_exports_every_declared_symbol():
    lib = gcx.load()
    for name in declared_symbols():
        assert hasattr(lib, name), name
    assert set(declared_symbols()) == set(gcx.SIGNATURES)


def test_version_and_strerror():
    assert gcx.gc_version() >= 100
    for st in (gcx.GC_OK, gcx.GC_EINVAL, gcx.GC_ELAUNCH, gcx.GC_ENOTSUP, 7):
        assert isinstance(gcx.strerror(st), str)


@pytest.mark.parametrize("m,s", [(1, 0), (3, 1), (6, 2), (20, 3), (50, 4), (100, 9), (200, 19), (9, 8)])
def test_assign_cyclic_matches_oracle(m, s):
    O, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_CYCLIC, m, m, s)
    assert (O == OA.cyclic_O(m, m, s)).all()
    o2, h2, p2 = OA.tables(OA.cyclic_O(m, m, s))
    assert (order == o2).all() and (holder == h2).all() and (hpos == p2).all()


def test_assign_from_order_matches_oracle():
    g = np.random.default_rng(0)
    for _ in range(30):
        N, m = g.integers(1, 12, size=2)
        A = g.random((N, m)) < 0.4
        O = np.zeros((N, m), dtype=np.int32)
        for j in range(m):
            rows = np.flatnonzero(A[:, j])
            g.shuffle(rows)
            O[rows, j] = np.arange(1, len(rows) + 1)
        delta = max(1, int((O != 0).sum(axis=0).max()))
        gamma = max(1, int((O != 0).sum(axis=1).max()))
        _, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_ORDER, N, m, -1, O, delta, gamma)
        o2, h2, p2 = OA.tables(O, delta, gamma)
        assert (order == o2).all() and (holder == h2).all() and (hpos == p2).all()


def _raw_assign(kind, N, m, s, O, delta, gamma):
    lib = gcx.load()
    order = np.zeros((m, max(delta, 1)), dtype=np.int32)
    holder = np.zeros((N, max(gamma, 1)), dtype=np.int32)
    hpos = np.zeros((N, max(gamma, 1)), dtype=np.int32)
    Op = O.ctypes.data if O is not None else None
    return lib.gc_assign(kind, N, m, s, Op, delta, gamma, order.ctypes.data, holder.ctypes.data,
                         hpos.ctypes.data)


def test_assign_rejects_bad_arguments():
    E = gcx.GC_EINVAL
    assert _raw_assign(gcx.GC_ASSIGN_CYCLIC, 5, 6, 1, None, 2, 2) == E      # N != m
    assert _raw_assign(gcx.GC_ASSIGN_CYCLIC, 5, 5, 5, None, 6, 6) == E      # s >= m
    assert _raw_assign(gcx.GC_ASSIGN_CYCLIC, 5, 5, 1, None, 3, 2) == E      # delta != s+1
    assert _raw_assign(7, 5, 5, 1, None, 2, 2) == E                          # unknown kind
    assert _raw_assign(gcx.GC_ASSIGN_ORDER, 3, 3, -1, None, 2, 2) == E       # O missing
    bad = np.array([[1, 0, 0], [1, 0, 0], [0, 0, 0]], dtype=np.int32)      # two chunks at position 1
    assert _raw_assign(gcx.GC_ASSIGN_ORDER, 3, 3, -1, bad, 3, 3) == E
    gap = np.array([[1, 0, 0], [3, 0, 0], [0, 0, 0]], dtype=np.int32)      # positions 1, 3: a gap
    assert _raw_assign(gcx.GC_ASSIGN_ORDER, 3, 3, -1, gap, 3, 3) == E
    narrow = np.array([[1, 1, 1], [0, 0, 0], [0, 0, 0]], dtype=np.int32)   # gamma 3 > table width 2
    assert _raw_assign(gcx.GC_ASSIGN_ORDER, 3, 3, -1, narrow, 1, 2) == E


def test_device_calls_validate_on_the_host():
    """Bad sizes and null pointers are rejected before any device work (no GPU needed)."""
    lib = gcx.load()
    E = gcx.GC_EINVAL
    p = 16  # a dummy non-null address; validation must fail before it is used
    assert lib.gc_decode_coeffs(p, 4, 6, 0, p, 3, p, p, 3, p, 1, p, p, p, p, None) == E       # m = 0
    assert lib.gc_decode_coeffs(p, 4, 6, 6, p, 3, p, p, 3, p, 9, p, p, p, p, None) == E       # ell > 8
    assert lib.gc_decode_coeffs(None, 4, 6, 6, p, 3, p, p, 3, p, 1, p, p, p, p, None) == E    # null psi
    assert lib.gc_decode_coeffs(p, 4, 6, 2000, p, 3, p, p, 3, p, 1, p, p, p, p, None) == E    # m too big
    assert lib.gc_decode_coeffs(p, -1, 6, 6, p, 3, p, p, 3, p, 1, p, p, p, p, None) == E      # P < 0
    assert lib.gc_decode_coeffs(p, 0, 6, 6, p, 3, p, p, 3, p, 1, p, p, p, p, None) == gcx.GC_OK  # P = 0
    assert lib.gc_encode(p, 5, 6, 64, p, p, p, 4, 6, 3, 1, p, None) == E                       # dtype
    assert lib.gc_encode(p, 0, 6, 0, p, p, p, 4, 6, 3, 1, p, None) == E                        # d = 0
    assert lib.gc_encode(None, 0, 6, 64, p, p, p, 4, 6, 3, 1, p, None) == E                    # null G
    assert lib.gc_encode(p, 0, 6, 64, p, p, p, 0, 6, 3, 1, p, None) == gcx.GC_OK                # P = 0
    assert lib.gc_reconstruct(p, p, p, 4, 6, 64, 0, p, None, None, None, 0, None) == E         # ell = 0
    assert lib.gc_reconstruct(p, p, p, 4, 6, 64, 1, p, None, p, None, 0, None) == E            # sqerr w/o gsum
    assert lib.gc_reconstruct(p, p, p, 4, 6, 1 << 20, 1, None, p, p, None, 0, None) == E       # workspace
    assert lib.gc_reconstruct(p, p, None, 4, 6, 64, 1, p, None, None, None, 0, None) == E      # null psi
    ws = gcx.gc_decode_direct_workspace_size(4, 6, 64, 1)
    args = dict(G=p, g_dtype=0, N=6, d=64, psi=p, P=4, m=6, delta=3, holder=p, hpos=p, gamma=3, R=p,
                ell=1, ghat=p, gsum=None, sqerr=None, ws=p, ws_bytes=ws, stream=None)

    def direct(**kw):
        return lib.gc_decode_direct(*{**args, **kw}.values())
    assert direct(ell=0) == E and direct(ell=9) == E and direct(g_dtype=3) == E
    assert direct(ghat=None) == E                                       # neither output
    assert direct(sqerr=p) == E                                         # sqerr without gsum
    assert direct(ws_bytes=ws - 1) == E and direct(ws=None) == E        # workspace
    assert direct(ws=p + 4) == E                                        # unaligned workspace
    assert direct(holder=None) == E and direct(G=None) == E
    assert direct(P=0) == gcx.GC_OK
    assert lib.gc_chunk_grads(p, p, p, 2, 3, 8, 1, 5, p, p, 1 << 20, None) == E                # loss
    assert lib.gc_chunk_grads(p, p, p, 2, 3, 8, 1, 0, p, p, 4, None) == E                      # small ws
    assert lib.gc_sum_chunks(p, 3, 2, 8, p, None) == E


def test_workspace_sizes():
    # fused single-pass path (d % 4 == 0, d <= 16384): two d-float partial slots per block
    assert gcx.gc_chunk_grads_workspace_size(50, 512, 16384, 1) == 4 * 512 * 2 * 16384
    # general path: one residual per sample row and point
    assert gcx.gc_chunk_grads_workspace_size(50, 512, 16385, 2) == 4 * 2 * 50 * 512
    # matrix cores (b >= 16 points): split-K partials of Z plus the residuals.  200 (b = 64)
    # or 400 (b = 256) output tiles of Z; 5 splits fill two whole rounds of 512 resident
    # blocks (4 or 8 splits would leave a last round 1/8 full)
    assert gcx.gc_chunk_grads_workspace_size(50, 512, 16384, 64) == 4 * (5 + 1) * 50 * 512 * 64
    assert gcx.gc_chunk_grads_workspace_size(50, 512, 16384, 256) == 4 * (5 + 1) * 50 * 512 * 256
    # one fp64 partial per (pattern, 4096-wide piece of a block), none when a block has one piece
    assert gcx.gc_reconstruct_workspace_size(10000, 50, 16384, 1) == 8 * 10000 * 4
    assert gcx.gc_reconstruct_workspace_size(10, 50, 4096, 1) == 0
    assert gcx.gc_reconstruct_workspace_size(10, 50, 4097, 1) == 8 * 10 * 2
    assert gcx.gc_reconstruct_workspace_size(10, 50, 16384, 4) == 0
    assert gcx.gc_reconstruct_workspace_size(10, 100, 1 << 20, 8) == 8 * 10 * 32
    # direct estimate: fp32 mixing rows padded to 32 columns (256-byte rounded), then one fp64
    # error partial per (row, 128-column tile)
    assert gcx.gc_decode_direct_workspace_size(10000, 50, 16384, 1) == 4 * 10000 * 64 + 8 * 10000 * 128
    assert gcx.gc_decode_direct_workspace_size(3, 6, 64, 3) == 1280 + 8 * 9  # 4*9*32 = 1152 -> 1280
    assert gcx.gc_decode_direct_workspace_size(0, 6, 64, 1) == 0


def test_assign_regular_algorithm2():
    """gc_assign(GC_ASSIGN_REGULAR): Algorithm 2 in the library gives a valid, optimal ordering
    (orderings are not unique; validity and Q_max are)."""
    import pins
    import oracle.ordering as OO
    from workloads import gen
    g = np.random.default_rng(5)
    supports = [pins._random_regular_support(g, m, dl) for m, dl in [(4, 2), (10, 3), (50, 5), (97, 9)]]
    supports.append(gen.random_regular_graph(200, 8) != 0)
    supports.append(OA.cyclic_O(20, 20, 3) != 0)
    for S in supports:
        m, delta = S.shape[0], int(S.sum(axis=0)[0])
        O, order, holder, hpos = gcx.gc_assign(gcx.GC_ASSIGN_REGULAR, m, m, -1, S.astype(np.int32), delta, delta)
        pins.check_ordering(O, S)
        assert OO.q_max(O) == OO.q_max(OO.chunk_ordering(S))
        o2, h2, p2 = OA.tables(O, delta, delta)
        assert (order == o2).all() and (holder == h2).all() and (hpos == p2).all()


def test_assign_regular_rejects_irregular():
    S = np.eye(5, dtype=np.int32)
    S[0, 1] = 1                                     # row 0 has degree 2
    assert _raw_assign(gcx.GC_ASSIGN_REGULAR, 5, 5, -1, S, 1, 1) == gcx.GC_EINVAL
    S2 = np.ones((4, 5), dtype=np.int32)          # N != m
    assert _raw_assign(gcx.GC_ASSIGN_REGULAR, 4, 5, -1, S2, 5, 4) == gcx.GC_EINVAL


def test_qmax_matches_the_oracle():
    """gc_qmax (the Sec. 3 ordering metric) against the oracle's direct count, on cyclic codes,
    random orderings of random regular supports, Algorithm 2 orderings (where every row of O
    sums to delta(delta+1)/2, so Q_max = delta(delta+1)/2 + (m - delta - 1) delta) and a
    non-square assignment; invalid orderings are rejected."""
    import oracle.ordering as OO
    import pins
    g = np.random.default_rng(21)
    for m, s in [(6, 2), (20, 3), (50, 4), (200, 7)]:
        O = OA.cyclic_O(m, m, s)
        Q, qm = gcx.gc_qmax(O)
        assert (Q == OA.Q(O)).all() and qm == OO.q_max(O)
    for m, delta in [(12, 3), (40, 5), (200, 8)]:
        S = pins._random_regular_support(g, m, delta)
        for _ in range(3):
            O = np.zeros((m, m), dtype=np.int64)
            for j in range(m):
                rows = np.flatnonzero(S[:, j])
                O[rows, j] = g.permutation(delta) + 1
            Q, qm = gcx.gc_qmax(O)
            assert (Q == OA.Q(O)).all() and qm == OO.q_max(O)
        O2, _, _, _ = gcx.gc_assign(gcx.GC_ASSIGN_REGULAR, m, m, -1, S.astype(np.int32), delta, delta)
        _, qm = gcx.gc_qmax(O2)
        assert qm == delta * (delta + 1) // 2 + (m - delta - 1) * delta
    O = pins.sec2_2_O()                           # unequal loads (the Sec. 2.2 example)
    assert (gcx.gc_qmax(O)[0] == OA.Q(O)).all()
    O = np.zeros((7, 5), dtype=np.int64)          # N = 7 chunks over m = 5 workers
    nxt = np.zeros(5, dtype=np.int64)
    for i in range(7):
        for j in (i % 5, (i + 2) % 5):
            nxt[j] += 1
            O[i, j] = nxt[j]
    assert (gcx.gc_qmax(O)[0] == OA.Q(O)).all()
    bad = OA.cyclic_O(6, 6, 2).copy()
    bad[0, 0] = 2                                  # two chunks at position 2 of worker 0
    with pytest.raises(gcx.GcxError):
        gcx.gc_qmax(bad)


def test_binding_shares_torchs_hip_runtime():
    """The binding loads libgcx.so after torch, so a process holds one HIP runtime (the
    one torch ships): loaded first, the library pulls in the system runtime and torch then
    maps its own next to it, and launches on torch's streams fail."""
    import subprocess
    import sys
    code = ("from paper_2405_19509_amd import gcx; gcx.load(); import torch; "
            "maps = open('/proc/self/maps').read().splitlines(); "
            "print(len({l.split()[-1] for l in maps if 'libamdhip64' in l}))")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip().splitlines()[-1] == "1"
