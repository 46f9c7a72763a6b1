"""Python binding of the gcx C ABI (include/gcx.h): argument marshalling only.

Every function here has the name of the C entry point it calls.  Device
arrays are torch tensors on the current HIP device (torch is used for device
memory and streams); each call checks dtype, device, contiguity and shape,
allocates outputs the caller did not pass, and enqueues the library's kernels
on torch's current stream.  No step of the hot path runs in Python or torch:
if libgcx.so is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

GC_OK, GC_EINVAL, GC_ELAUNCH, GC_ENOTSUP, GC_ESCRATCH = 0, -1, -2, -3, -4
GC_NOALLOC_SCRATCH_BYTES = 4 << 20
GC_ASSIGN_CYCLIC, GC_ASSIGN_ORDER, GC_ASSIGN_REGULAR = 0, 1, 2
GC_LOSS_LINEAR, GC_LOSS_LOGISTIC = 0, 1
GC_F32, GC_BF16 = 0, 1
GC_DEC_NO, GC_DEC_YES, GC_DEC_INVALID = 0, 1, 2
GC_MAX_ELL = 8
GC_MAX_M = 1024
GC_MAX_DELTA = 64

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgcx.so")

# every symbol the header declares, with (restype, argtypes)
_c = ctypes
_p = _c.c_void_p
_i32, _i64, _sz = _c.c_int32, _c.c_int64, _c.c_size_t
SIGNATURES = {
    "gc_version": (_c.c_int, []),
    "gc_strerror": (_c.c_char_p, [_c.c_int]),
    "gc_assign": (_c.c_int, [_i32, _i32, _i32, _i32, _p, _i32, _i32, _p, _p, _p]),
    "gc_qmax": (_c.c_int, [_p, _i32, _i32, _p, _p]),
    "gc_chunk_grads_workspace_size": (_sz, [_i32, _i32, _i64, _i32]),
    "gc_chunk_grads": (_c.c_int, [_p, _p, _p, _i32, _i32, _i64, _i32, _i32, _p, _p, _sz, _p]),
    "gc_sum_chunks": (_c.c_int, [_p, _i32, _i32, _i64, _p, _p]),
    "gc_decode_coeffs": (_c.c_int, [_p, _i64, _i32, _i32, _p, _i32, _p, _p, _i32, _p, _i32,
                                    _p, _p, _p, _p, _p]),
    "gc_encode": (_c.c_int, [_p, _i32, _i32, _i64, _p, _p, _p, _i64, _i32, _i32, _i32, _p, _p]),
    "gc_progress": (_c.c_int, [_p, _p, _i64, _i32, _i32, _p, _i32, _p, _p]),
    "gc_completion_times": (_c.c_int, [_p, _p, _i64, _i32, _i32, _i32, _p, _p, _i32, _i32, _p, _p, _p]),
    "gc_original_ls": (_c.c_int, [_p, _i64, _i32, _i32, _p, _i32, _p, _i32, _i32, _c.c_double, _p, _p, _p]),
    "gc_reconstruct_workspace_size": (_sz, [_i64, _i32, _i64, _i32]),
    "gc_reconstruct": (_c.c_int, [_p, _p, _p, _i64, _i32, _i64, _i32, _p, _p, _p, _p, _sz, _p]),
    "gc_reconstruct_noalloc": (_c.c_int, [_p, _p, _p, _i64, _i32, _i64, _i32, _p, _p, _p, _p]),
    "gc_decode_direct_workspace_size": (_sz, [_i64, _i32, _i64, _i32]),
    "gc_decode_direct": (_c.c_int, [_p, _i32, _i32, _i64, _p, _i64, _i32, _i32, _p, _p, _i32, _p,
                                    _i32, _p, _p, _p, _p, _sz, _p]),
}

_lib = None


class GcxError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {status} ({strerror(status)})")


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libgcx.so (once).  Raises if it has not been built.

    torch is imported first: the PyTorch ROCm wheel ships its own HIP runtime, and the
    library must bind to that one (the one that owns torch's memory and streams).  Loaded
    before torch, libgcx.so would pull in the system HIP runtime and torch would then load
    its own, two runtimes in one process, and launches on torch's streams would fail."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2405_19509_amd.build`")
    try:
        import torch  # noqa: F401  (see above: before the library, for its HIP runtime)
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def strerror(status: int) -> str:
    return load().gc_strerror(status).decode()


def gc_version() -> int:
    return load().gc_version()


def _check(fn: str, st: int) -> None:
    if st != GC_OK:
        raise GcxError(fn, st)


def _torch():
    import torch
    return torch


def _stream(stream) -> int:
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream)


def _dev(t, name, dtype, shape=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t.data_ptr()


def _g_dtype(G):
    torch = _torch()
    if G.dtype == torch.float32:
        return GC_F32
    if G.dtype == torch.bfloat16:
        return GC_BF16
    raise ValueError("chunk gradients must be float32 or bfloat16")


# ---------------------------------------------------------------------------

def gc_assign(kind: int, N: int, m: int, s: int = -1, O: Optional[np.ndarray] = None,
              delta: Optional[int] = None, gamma: Optional[int] = None):
    """Host call.  Returns (O, order, holder, hpos) as int32 numpy arrays.  For
    GC_ASSIGN_REGULAR, O is the support on input and the returned O the ordering."""
    lib = load()
    if kind == GC_ASSIGN_CYCLIC:
        delta = s + 1 if delta is None else delta
        gamma = s + 1 if gamma is None else gamma
        O = np.zeros((N, m), dtype=np.int32)
    else:
        if O is None:
            raise ValueError("GC_ASSIGN_ORDER needs O")
        O = np.ascontiguousarray(O, dtype=np.int32)
        if O.shape != (N, m):
            raise ValueError("O must be [N][m]")
        delta = int((O != 0).sum(axis=0).max()) if delta is None else delta
        gamma = int((O != 0).sum(axis=1).max()) if gamma is None else gamma
    order = np.zeros((m, max(delta, 0)), dtype=np.int32)
    holder = np.zeros((N, max(gamma, 0)), dtype=np.int32)
    hpos = np.zeros((N, max(gamma, 0)), dtype=np.int32)
    st = lib.gc_assign(kind, N, m, s, O.ctypes.data, delta, gamma, order.ctypes.data,
                       holder.ctypes.data, hpos.ctypes.data)
    _check("gc_assign", st)
    return O, order, holder, hpos


def gc_qmax(O):
    """O [N][m] ordering matrix (host) -> (Q [N] int64, Q_max): the Sec. 3 metric."""
    O = np.ascontiguousarray(O, dtype=np.int32)
    N, m = O.shape
    Q = np.empty(N, dtype=np.int64)
    qmax = ctypes.c_int64(0)
    _check("gc_qmax", load().gc_qmax(O.ctypes.data, N, m, Q.ctypes.data, ctypes.byref(qmax)))
    return Q, int(qmax.value)


def gc_chunk_grads_workspace_size(N: int, n: int, d: int, b: int) -> int:
    return int(load().gc_chunk_grads_workspace_size(N, n, d, b))


def gc_chunk_grads(X, y, W, loss: int, G=None, workspace=None, stream=None):
    """X [N][n][d], y [N][n], W [d] or [b][d] fp32 -> G [N][d] or [b][N][d] fp32."""
    torch = _torch()
    lib = load()
    N, n, d = X.shape
    single = W.dim() == 1
    b = 1 if single else W.shape[0]
    gshape = (N, d) if single else (b, N, d)
    if G is None:
        G = torch.empty(gshape, dtype=torch.float32, device=X.device)
    need = gc_chunk_grads_workspace_size(N, n, d, b)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=X.device)
    st = lib.gc_chunk_grads(_dev(X, "X", torch.float32), _dev(y, "y", torch.float32, (N, n)),
                            _dev(W, "W", torch.float32, (d,) if single else (b, d)), N, n, d, b, loss,
                            _dev(G, "G", torch.float32, gshape),
                            _dev(workspace, "workspace", torch.uint8), workspace.numel(),
                            _stream(stream))
    _check("gc_chunk_grads", st)
    return G


def gc_sum_chunks(G, gsum=None, stream=None):
    """G [N][d] (fp32 or bf16) -> gsum [d] fp32."""
    torch = _torch()
    N, d = G.shape
    if gsum is None:
        gsum = torch.empty(d, dtype=torch.float32, device=G.device)
    st = load().gc_sum_chunks(_dev(G, "G", G.dtype), _g_dtype(G), N, d,
                              _dev(gsum, "gsum", torch.float32, (d,)), _stream(stream))
    _check("gc_sum_chunks", st)
    return gsum


def gc_decode_coeffs(psi, order, holder, hpos, R, cov=None, dec=None, coef_err=None, Bc=None,
                     coverage_only: bool = False, stream=None):
    """psi [P][m] int32, tables from gc_assign (device int32), R [ell][m] fp32
    -> (cov [P][N] int32, dec [P] uint8, coef_err [P] int32, Bc [P][m][delta][ell] fp32).
    coverage_only: skip the coefficient solves (Bc is returned as None)."""
    torch = _torch()
    P, m = psi.shape
    m2, delta = order.shape
    N, gamma = holder.shape
    ell = R.shape[0]
    if m2 != m or R.shape[1] != m:
        raise ValueError("psi, order and R disagree on m")
    dv = psi.device
    if cov is None:
        cov = torch.empty((P, N), dtype=torch.int32, device=dv)
    if dec is None:
        dec = torch.empty(P, dtype=torch.uint8, device=dv)
    if coef_err is None:
        coef_err = torch.empty(P, dtype=torch.int32, device=dv)
    if Bc is None and not coverage_only:
        Bc = torch.empty((P, m, delta, ell), dtype=torch.float32, device=dv)
    st = load().gc_decode_coeffs(
        _dev(psi, "psi", torch.int32), P, N, m, _dev(order, "order", torch.int32), delta,
        _dev(holder, "holder", torch.int32), _dev(hpos, "hpos", torch.int32, (N, gamma)), gamma,
        _dev(R, "R", torch.float32), ell, _dev(cov, "cov", torch.int32, (P, N)),
        _dev(dec, "dec", torch.uint8, (P,)), _dev(coef_err, "coef_err", torch.int32, (P,)),
        _dev(Bc, "Bc", torch.float32, (P, m, delta, ell)) if Bc is not None else None, _stream(stream))
    _check("gc_decode_coeffs", st)
    return cov, dec, coef_err, Bc


def gc_encode(G, psi, order, Bc, T=None, stream=None):
    """G [N][d] (fp32 or bf16), psi [P][m], order [m][delta], Bc [P][m][delta][ell]
    -> T [P][m][L] fp32, L = ceil(d / ell)."""
    torch = _torch()
    N, d = G.shape
    P, m, delta, ell = Bc.shape
    L = -(-d // ell)
    if T is None:
        T = torch.empty((P, m, L), dtype=torch.float32, device=G.device)
    st = load().gc_encode(_dev(G, "G", G.dtype), _g_dtype(G), N, d,
                          _dev(psi, "psi", torch.int32, (P, m)),
                          _dev(order, "order", torch.int32, (m, delta)),
                          _dev(Bc, "Bc", torch.float32), P, m, delta, ell,
                          _dev(T, "T", torch.float32, (P, m, L)), _stream(stream))
    _check("gc_encode", st)
    return T


def gc_reconstruct_workspace_size(P: int, m: int, d: int, ell: int) -> int:
    return int(load().gc_reconstruct_workspace_size(P, m, d, ell))


def gc_reconstruct(T, R, d: int, psi, ghat=None, gsum=None, sqerr=None, want_ghat: bool = True,
                   workspace=None, stream=None):
    """T [P][m][L], R [ell][m], psi [P][m] (required: rows with psi <= 0 are not read) ->
    (ghat [P][d] or None, sqerr [P] fp64 or None).  sqerr is computed when gsum [d] is given."""
    torch = _torch()
    P, m, L = T.shape
    ell = R.shape[0]
    if L != -(-d // ell):
        raise ValueError("T's row length does not match ceil(d / ell)")
    dv = T.device
    if want_ghat and ghat is None:
        ghat = torch.empty((P, d), dtype=torch.float32, device=dv)
    if gsum is not None and sqerr is None:
        sqerr = torch.empty(P, dtype=torch.float64, device=dv)
    ws_ptr, ws_bytes = None, 0
    if sqerr is not None:
        need = gc_reconstruct_workspace_size(P, m, d, ell)
        if need and workspace is None:
            workspace = torch.empty(need, dtype=torch.uint8, device=dv)
        if workspace is not None:
            ws_ptr, ws_bytes = _dev(workspace, "workspace", torch.uint8), workspace.numel()
    st = load().gc_reconstruct(
        _dev(T, "T", torch.float32), _dev(R, "R", torch.float32, (ell, m)),
        _dev(psi, "psi", torch.int32, (P, m)), P, m, d, ell,
        _dev(ghat, "ghat", torch.float32, (P, d)) if ghat is not None else None,
        _dev(gsum, "gsum", torch.float32, (d,)) if gsum is not None else None,
        _dev(sqerr, "sqerr", torch.float64, (P,)) if sqerr is not None else None,
        ws_ptr, ws_bytes, _stream(stream))
    _check("gc_reconstruct", st)
    return ghat, sqerr


def gc_reconstruct_noalloc(T, R, d: int, psi, ghat, gsum=None, sqerr=None, stream=None):
    """gc_reconstruct without a workspace: the library's fixed per-device scratch array holds
    the squared error's partial sums.  Outputs must be passed in (ghat [P][d] or None; sqerr
    [P] fp64 with gsum [d], or None); nothing is allocated here.  Returns (ghat, sqerr)."""
    torch = _torch()
    P, m, L = T.shape
    ell = R.shape[0]
    if L != -(-d // ell):
        raise ValueError("T's row length does not match ceil(d / ell)")
    st = load().gc_reconstruct_noalloc(
        _dev(T, "T", torch.float32), _dev(R, "R", torch.float32, (ell, m)),
        _dev(psi, "psi", torch.int32, (P, m)), P, m, d, ell,
        _dev(ghat, "ghat", torch.float32, (P, d)) if ghat is not None else None,
        _dev(gsum, "gsum", torch.float32, (d,)) if gsum is not None else None,
        _dev(sqerr, "sqerr", torch.float64, (P,)) if sqerr is not None else None, _stream(stream))
    _check("gc_reconstruct_noalloc", st)
    return ghat, sqerr


def gc_decode_direct_workspace_size(P: int, N: int, d: int, ell: int) -> int:
    return int(load().gc_decode_direct_workspace_size(P, N, d, ell))


def gc_decode_direct(G, psi, order, holder, hpos, R, ghat=None, gsum=None, sqerr=None,
                     want_ghat: bool = True, workspace=None, stream=None):
    """G [N][d] (fp32 or bf16), psi [P][m], tables from gc_assign, R [ell][m] ->
    (ghat [P][d] or None, sqerr [P] fp64 or None): the estimate of gc_reconstruct formed from
    the chunk gradients directly.  sqerr is computed when gsum [d] is given."""
    torch = _torch()
    N, d = G.shape
    P, m = psi.shape
    ell = R.shape[0]
    delta = order.shape[1]
    gamma = holder.shape[1]
    dv = G.device
    if want_ghat and ghat is None:
        ghat = torch.empty((P, d), dtype=torch.float32, device=dv)
    if gsum is not None and sqerr is None:
        sqerr = torch.empty(P, dtype=torch.float64, device=dv)
    need = gc_decode_direct_workspace_size(P, N, d, ell)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dv)
    st = load().gc_decode_direct(
        _dev(G, "G", G.dtype), _g_dtype(G), N, d, _dev(psi, "psi", torch.int32, (P, m)), P, m, delta,
        _dev(holder, "holder", torch.int32, (N, gamma)), _dev(hpos, "hpos", torch.int32, (N, gamma)),
        gamma, _dev(R, "R", torch.float32, (ell, m)), ell,
        _dev(ghat, "ghat", torch.float32, (P, d)) if ghat is not None else None,
        _dev(gsum, "gsum", torch.float32, (d,)) if gsum is not None else None,
        _dev(sqerr, "sqerr", torch.float64, (P,)) if sqerr is not None else None,
        _dev(workspace, "workspace", torch.uint8), workspace.numel(), _stream(stream))
    _check("gc_decode_direct", st)
    return ghat, sqerr


def gc_progress(tau, T, failed=None, psi=None, stream=None):
    """tau [R][m][delta] fp64, T [G] fp64, failed [R][m] uint8 or None -> psi [R][G][m] int32."""
    torch = _torch()
    R, m, delta = tau.shape
    G = T.shape[0]
    if psi is None:
        psi = torch.empty((R, G, m), dtype=torch.int32, device=tau.device)
    st = load().gc_progress(_dev(tau, "tau", torch.float64),
                            _dev(failed, "failed", torch.uint8, (R, m)) if failed is not None else None,
                            R, m, delta, _dev(T, "T", torch.float64, (G,)), G,
                            _dev(psi, "psi", torch.int32, (R, G, m)), _stream(stream))
    _check("gc_progress", st)
    return psi


def gc_completion_times(tau, holder, hpos, ell: int, failed=None, partial=None, original=None,
                        stream=None):
    """tau [R][m][delta] fp64, tables from gc_assign -> (partial [R], original [R]) fp64."""
    torch = _torch()
    R, m, delta = tau.shape
    N, gamma = holder.shape
    if partial is None:
        partial = torch.empty(R, dtype=torch.float64, device=tau.device)
    if original is None:
        original = torch.empty(R, dtype=torch.float64, device=tau.device)
    st = load().gc_completion_times(
        _dev(tau, "tau", torch.float64),
        _dev(failed, "failed", torch.uint8, (R, m)) if failed is not None else None, R, N, m, delta,
        _dev(holder, "holder", torch.int32), _dev(hpos, "hpos", torch.int32, (N, gamma)), gamma, ell,
        _dev(partial, "partial", torch.float64, (R,)), _dev(original, "original", torch.float64, (R,)),
        _stream(stream))
    _check("gc_completion_times", st)
    return partial, original


def gc_original_ls(psi, order, holder, max_iter: int = 1000, tol: float = 1e-12, err=None,
                   iters=None, stream=None):
    """psi [P][m] int32, tables -> (err [P] fp64, iters [P] int32): original GC's
    least-squares error over the fully finished workers."""
    torch = _torch()
    P, m = psi.shape
    _, delta = order.shape
    N, gamma = holder.shape
    if err is None:
        err = torch.empty(P, dtype=torch.float64, device=psi.device)
    if iters is None:
        iters = torch.empty(P, dtype=torch.int32, device=psi.device)
    st = load().gc_original_ls(_dev(psi, "psi", torch.int32), P, N, m,
                               _dev(order, "order", torch.int32, (m, delta)), delta,
                               _dev(holder, "holder", torch.int32, (N, gamma)), gamma, max_iter, tol,
                               _dev(err, "err", torch.float64, (P,)),
                               _dev(iters, "iters", torch.int32, (P,)), _stream(stream))
    _check("gc_original_ls", st)
    return err, iters
