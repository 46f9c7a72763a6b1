"""gc_reconstruct_noalloc (the combine with its scratch in the library's fixed device array)
against gc_reconstruct (caller workspace): identical estimates and squared errors on two calls
in a row, the second smaller, so the second reads only partial sums it wrote itself."""
from __future__ import annotations

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2405_19509_amd import gcx  # noqa: E402

# (patterns, workers, d, ell): the first spans 64 pieces per pattern (6,144 partial sums) on
# the float4 path, the second 3 pieces on the scalar path (L = 6667 is not a multiple of 4)
CALLS = [(96, 16, 1 << 18, 1), (10, 16, 20001, 3)]


def inputs(P, m, d, ell, seed):
    rng = np.random.default_rng(seed)
    L = -(-d // ell)
    T = rng.standard_normal((P, m, L), dtype=np.float32)
    R = rng.standard_normal((ell, m), dtype=np.float32)
    psi = rng.integers(0, 4, size=(P, m), dtype=np.int32)   # about a quarter of the rows: stragglers
    gsum = rng.standard_normal(d, dtype=np.float32)
    return [torch.from_numpy(a).cuda() for a in (T, R, psi, gsum)]


def test_noalloc_matches_workspace_call_twice():
    for call, (P, m, d, ell) in enumerate(CALLS):
        print(f"call {call}: P={P} m={m} d={d} ell={ell}", flush=True)
        assert gcx.gc_reconstruct_workspace_size(P, m, d, ell) <= gcx.GC_NOALLOC_SCRATCH_BYTES
        T, R, psi, gsum = inputs(P, m, d, ell, seed=call)
        ref_gh, ref_se = gcx.gc_reconstruct(T, R, d, psi, gsum=gsum)
        gh = torch.full((P, d), float("nan"), device="cuda")
        se = torch.full((P,), float("nan"), dtype=torch.float64, device="cuda")
        gcx.gc_reconstruct_noalloc(T, R, d, psi, gh, gsum=gsum, sqerr=se)
        torch.cuda.synchronize()
        assert torch.equal(gh, ref_gh)
        assert torch.equal(se, ref_se)
        # error-only mode: the same squared errors
        se2 = torch.full((P,), float("nan"), dtype=torch.float64, device="cuda")
        gcx.gc_reconstruct_noalloc(T, R, d, psi, None, gsum=gsum, sqerr=se2)
        torch.cuda.synchronize()
        assert torch.equal(se2, ref_se)
        # and they are the squared errors of the returned estimate
        direct = ((gh.double() - gsum.double()) ** 2).sum(dim=1)
        assert torch.allclose(se, direct, rtol=1e-10, atol=0)


def test_noalloc_rejects_oversized_request():
    P, m, d, ell = 1000, 4, 1 << 24, 1
    assert gcx.gc_reconstruct_workspace_size(P, m, d, ell) > gcx.GC_NOALLOC_SCRATCH_BYTES
    p = 16  # never dereferenced: the size check comes first
    st = gcx.load().gc_reconstruct_noalloc(p, p, p, P, m, d, ell, None, p, p, None)
    assert st == gcx.GC_ESCRATCH
