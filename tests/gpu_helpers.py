"""Shared helpers for the GPU parity tests (HIP path vs the fp64 oracle)."""
import numpy as np
import torch

from oracle import recurrent
from paper_2606_08804_amd import qdelta, synth

f64 = synth.to_f64
TOL = {"f32": 1e-4, "bf16": 2e-2}


def normwise(got, ref):
    """max|got - ref| / max|ref| (absolute when the reference is all zero)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = np.abs(ref).max() if ref.size else 0.0
    err = np.abs(got - ref).max() if ref.size else 0.0
    return err / scale if scale > 0 else err


def dev(t):
    return None if t is None else t.cuda()


def gpu_fwd(d, save_states=False):
    o, Sf, saved = qdelta.chunk_fwd(dev(d["q"]), dev(d["k"]), dev(d["v"]), dev(d["beta"]),
                                    dev(d["lam"]), dev(d["log_alpha"]), dev(d["initial_state"]),
                                    cu_seqlens=dev(d["cu_seqlens"]), save_states=save_states)
    torch.cuda.synchronize()
    return o, Sf, saved


def gpu_bwd(d, saved=None, d_final_state=None):
    g = qdelta.chunk_bwd(dev(d["q"]), dev(d["k"]), dev(d["v"]), dev(d["beta"]), dev(d["lam"]),
                         dev(d["log_alpha"]), dev(d["initial_state"]), saved, dev(d["d_o"]),
                         d_final_state=dev(d_final_state), cu_seqlens=dev(d["cu_seqlens"]))
    torch.cuda.synchronize()
    return g


def _packed(d, key):
    x = f64(d[key])
    return None if x is None else (x[0] if d["cu_seqlens"] is not None else x)


def oracle_fwd(d):
    cu = d["cu_seqlens"]
    return recurrent.fwd(_packed(d, "q"), _packed(d, "k"), _packed(d, "v"), _packed(d, "beta"),
                         _packed(d, "lam"), _packed(d, "log_alpha"), f64(d["initial_state"]),
                         cu_seqlens=None if cu is None else cu.numpy())


def oracle_bwd(d, d_final_state=None):
    cu = d["cu_seqlens"]
    return recurrent.bwd(_packed(d, "q"), _packed(d, "k"), _packed(d, "v"), _packed(d, "beta"),
                         _packed(d, "lam"), _packed(d, "log_alpha"), f64(d["initial_state"]),
                         d_o=_packed(d, "d_o"), d_final_state=f64(d_final_state),
                         cu_seqlens=None if cu is None else cu.numpy())


def fwd_errors(d, o, Sf):
    o_ref, S_ref = oracle_fwd(d)
    og = f64(o.cpu())
    if d["cu_seqlens"] is not None:
        og = og[0]
    return dict(o=normwise(og, o_ref), final_state=normwise(f64(Sf.cpu()), S_ref))


def bwd_errors(d, g, d_final_state=None, skip=()):
    ref = oracle_bwd(d, d_final_state)
    out = {}
    for key in ("dq", "dk", "dv", "dbeta", "dlam", "dlog_alpha", "d_initial_state"):
        if key in skip:
            continue
        if ref[key] is None:
            assert g[key] is None
            continue
        got = f64(g[key].cpu())
        if d["cu_seqlens"] is not None and key != "d_initial_state":
            got = got[0]
        out[key] = normwise(got, ref[key])
    return out


def select_heads(d, heads):
    """Restrict a batch to a subset of heads (for oracle cost at full size)."""
    out = dict(d)
    for key in ("q", "k", "v", "beta", "lam", "log_alpha", "d_o"):
        if d[key] is not None:
            out[key] = d[key][:, :, heads].contiguous()
    if d["initial_state"] is not None:
        out["initial_state"] = d["initial_state"][:, heads].contiguous()
    return out
