"""fp64 token-by-token Q-Delta recurrence and its BPTT gradient (C, threaded).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper reference: Sec. 3.3, Eq. (qdelta_decay) with the mixed input
x_t = k_t + lambda_t q_t of Eq. (qdelta_gated_form):

    S_t = alpha_t S_{t-1} (I - beta_t x_t k_t^T) + beta_t v_t k_t^T,   o_t = S_t q_t.

The decay enters this module as log(alpha) (float32 values, widened exactly
to fp64, then alpha = exp(log alpha) in fp64), because the GPU boundary takes
log(alpha).  The gradient reported for it is d/d(log alpha) = alpha * d/d(alpha).

Layouts: dense ``[B, T, H, D]`` arrays, or packed ``[Ttot, H, D]`` arrays with
``cu_seqlens`` (int, length N+1).  Gates are ``[..., H]``.  States are
``[N, H, dv, dk]`` (row = value component).
"""
import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        path = _build.build(force=False)
        lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        lib.qdref_fwd.argtypes = [ctypes.c_int, P, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                  P, P, P, P, P, P, P, P, P, ctypes.c_int]
        lib.qdref_fwd.restype = ctypes.c_int
        lib.qdref_bwd.argtypes = [ctypes.c_int, P, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                  P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, ctypes.c_int]
        lib.qdref_bwd.restype = ctypes.c_int
        _LIB = lib
    return _LIB


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def _f64(a):
    return None if a is None else np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _pack(q, k, v, beta, lam, log_alpha, cu_seqlens, alpha=None):
    """Return packed fp64 arrays plus cu (int64) and the dense batch shape.

    ``alpha`` (the decay itself) may be given instead of ``log_alpha``."""
    q, k, v, beta, lam, log_alpha, alpha = map(_f64, (q, k, v, beta, lam, log_alpha, alpha))
    if alpha is not None and log_alpha is not None:
        raise ValueError("give log_alpha or alpha, not both")
    dense_shape = None
    if cu_seqlens is None:
        B, T, H, dk = q.shape
        dense_shape = (B, T)
        cu = np.arange(B + 1, dtype=np.int64) * T
        q, k = q.reshape(B * T, H, dk), k.reshape(B * T, H, dk)
        v = v.reshape(B * T, H, v.shape[-1])
        beta, lam = beta.reshape(B * T, H), lam.reshape(B * T, H)
        if log_alpha is not None:
            log_alpha = log_alpha.reshape(B * T, H)
        if alpha is not None:
            alpha = alpha.reshape(B * T, H)
    else:
        cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int64))
    if log_alpha is not None:
        alpha = np.exp(log_alpha)
    return q, k, v, beta, lam, alpha, cu, dense_shape


def fwd(q, k, v, beta, lam, log_alpha=None, initial_state=None, cu_seqlens=None,
        nthreads=None, alpha=None):
    """Run the recurrence.  Returns ``(o, final_state)`` in fp64."""
    q, k, v, beta, lam, alpha, cu, dense = _pack(q, k, v, beta, lam, log_alpha, cu_seqlens,
                                                 alpha)
    Ttot, H, dk = q.shape
    dv = v.shape[-1]
    N = len(cu) - 1
    S0 = _f64(initial_state)
    if S0 is not None:
        S0 = S0.reshape(N, H, dv, dk)
    o = np.zeros((Ttot, H, dv))
    Sf = np.zeros((N, H, dv, dk))
    rc = _lib().qdref_fwd(N, _ptr(cu), H, dk, dv, _ptr(q), _ptr(k), _ptr(v), _ptr(beta),
                          _ptr(lam), _ptr(alpha), _ptr(S0), _ptr(o), _ptr(Sf),
                          nthreads or default_threads())
    if rc != 0:
        raise ValueError("qdref_fwd rejected its arguments")
    if dense is not None:
        o = o.reshape(dense[0], dense[1], H, dv)
    return o, Sf


def bwd(q, k, v, beta, lam, log_alpha=None, initial_state=None, d_o=None,
        d_final_state=None, cu_seqlens=None, nthreads=None, alpha=None):
    """Exact gradients of <dO, o> + <dS_final, S_T>.

    Returns a dict with keys dq, dk, dv, dbeta, dlam, dlog_alpha (None when
    no decay is given), dalpha (gradient with respect to alpha itself, None
    when no decay is given) and d_initial_state.
    """
    q, k, v, beta, lam, alpha, cu, dense = _pack(q, k, v, beta, lam, log_alpha, cu_seqlens,
                                                 alpha)
    Ttot, H, dk = q.shape
    dv = v.shape[-1]
    N = len(cu) - 1
    S0 = _f64(initial_state)
    if S0 is not None:
        S0 = S0.reshape(N, H, dv, dk)
    dO = _f64(d_o)
    if dO is not None:
        dO = dO.reshape(Ttot, H, dv)
    dSf = _f64(d_final_state)
    if dSf is not None:
        dSf = dSf.reshape(N, H, dv, dk)
    dq = np.zeros_like(q)
    dk_ = np.zeros_like(k)
    dv_ = np.zeros_like(v)
    dbeta = np.zeros((Ttot, H))
    dlam = np.zeros((Ttot, H))
    dalpha = np.zeros((Ttot, H)) if alpha is not None else None
    dS0 = np.zeros((N, H, dv, dk))
    rc = _lib().qdref_bwd(N, _ptr(cu), H, dk, dv, _ptr(q), _ptr(k), _ptr(v), _ptr(beta),
                          _ptr(lam), _ptr(alpha), _ptr(S0), _ptr(dO), _ptr(dSf),
                          _ptr(dq), _ptr(dk_), _ptr(dv_), _ptr(dbeta), _ptr(dlam),
                          _ptr(dalpha), _ptr(dS0), nthreads or default_threads())
    if rc != 0:
        raise ValueError("qdref_bwd rejected its arguments")
    dla = None if alpha is None else alpha * dalpha
    out = dict(dq=dq, dk=dk_, dv=dv_, dbeta=dbeta, dlam=dlam, dlog_alpha=dla,
               dalpha=dalpha, d_initial_state=dS0)
    if dense is not None:
        B, T = dense
        for key in ("dq", "dk", "dv"):
            out[key] = out[key].reshape(B, T, H, -1)
        for key in ("dbeta", "dlam", "dlog_alpha", "dalpha"):
            if out[key] is not None:
                out[key] = out[key].reshape(B, T, H)
    return out
