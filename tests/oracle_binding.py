"""A stand-in for the library binding's chunk_fwd / chunk_bwd, computed by the
fp64 oracle on the CPU (and its row normalisation, from its definition), for tests of the autograd layer: its gradient wiring
on the CPU, and the reference that the GPU layer is compared with.

Same call signatures as ``paper_2606_08804_amd.qdelta``; results come back as
CPU tensors in the inputs' dtype.  ``saved`` is a token that carries nothing:
the oracle's backward recomputes the recurrence."""
import numpy as np
import torch

from oracle import recurrent


def _np(t):
    return None if t is None else t.detach().cpu().double().numpy()


def _packed(t, cu):
    a = _np(t)
    return None if a is None else (a[0] if cu is not None else a)


def _zeros_like_gate(beta):
    return np.zeros(beta.shape)


def _lam(lam, beta, cu):
    """Per-token lambda as an fp64 array: a tensor as is, a number broadcast
    to every token and head, None as zero."""
    if lam is None:
        return _zeros_like_gate(_packed(beta, cu))
    if isinstance(lam, (int, float)):
        return np.full(_packed(beta, cu).shape, float(lam))
    return _packed(lam, cu)


def chunk_fwd(q, k, v, beta, lam, log_alpha=None, initial_state=None, cu_seqlens=None,
              output_final_state=True, save_states=False, workspace=None):
    cu = None if cu_seqlens is None else cu_seqlens.cpu().numpy()
    lam_ = _lam(lam, beta, cu)
    o, Sf = recurrent.fwd(_packed(q, cu), _packed(k, cu), _packed(v, cu), _packed(beta, cu), lam_,
                          _packed(log_alpha, cu), _np(initial_state), cu_seqlens=cu)
    if cu is not None:
        o = o[None]
    o = torch.from_numpy(o).to(q.dtype)
    Sf = torch.from_numpy(Sf).to(torch.float32 if q.dtype != torch.float64 else q.dtype)
    saved = torch.zeros(1, dtype=torch.uint8) if save_states else None
    return o, (Sf if output_final_state else None), saved


def chunk_bwd(q, k, v, beta, lam, log_alpha, initial_state, saved_states, d_o,
              d_final_state=None, cu_seqlens=None, need_d_initial_state=True, workspace=None):
    cu = None if cu_seqlens is None else cu_seqlens.cpu().numpy()
    lam_ = _lam(lam, beta, cu)
    g = recurrent.bwd(_packed(q, cu), _packed(k, cu), _packed(v, cu), _packed(beta, cu), lam_,
                      _packed(log_alpha, cu), _np(initial_state), d_o=_packed(d_o, cu),
                      d_final_state=_np(d_final_state), cu_seqlens=cu)
    out = {}
    if isinstance(lam, (int, float)):
        # a constant lambda: one gradient, the sum over every token and head
        g = dict(g, dlam=np.asarray(g["dlam"].sum()))
        lam = torch.zeros((), dtype=beta.dtype)
    like = dict(dq=q, dk=k, dv=v, dbeta=beta, dlam=lam, dlog_alpha=log_alpha,
                d_initial_state=initial_state)
    for key, ref in like.items():
        if ref is None or g[key] is None or (key == "d_initial_state" and not need_d_initial_state):
            out[key] = None
            continue
        packed_rows = cu is not None and key != "d_initial_state" and np.ndim(g[key]) > 0
        a = g[key][None] if packed_rows else g[key]
        out[key] = torch.from_numpy(np.ascontiguousarray(a)).to(ref.dtype)
    return out


def l2norm_fwd(x):
    """The row normalisation's definition (same clamp and rnorm convention)."""
    n = x.norm(dim=-1)
    clamped = ~(n > 1e-12)
    r = 1.0 / torch.where(clamped, torch.full_like(n, 1e-12), n)
    return x * r[..., None], torch.where(clamped, -r, r)


def l2norm_bwd(y, rn, dy):
    r = rn.abs()[..., None]
    proj = torch.where(rn > 0, (y * dy).sum(-1), torch.zeros_like(rn))[..., None]
    return r * (dy - y * proj)
