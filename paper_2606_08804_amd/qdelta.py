"""Python binding of libqdelta.so (ctypes).  Argument marshalling only.

PyTorch supplies device memory and the current HIP stream; every step of the
Q-Delta computation runs in the library's HIP kernels.  There is no fallback:
if ``libqdelta.so`` is missing or fails to load, every entry point raises.

Functions mirror the C ABI in ``include/qdelta.h``:

chunk_fwd(q, k, v, beta, lam, log_alpha=None, initial_state=None, cu_seqlens=None,
          output_final_state=True, save_states=False) -> (o, final_state, saved)
          (saved: uint8 device buffer holding the saved context for the backward)
chunk_fwd_noalloc(q, k, v, beta, lam, log_alpha=None, initial_state=None, out=None,
          final_state_out=None) -> (o, final_state)    (dense; library-owned scratch, no workspace)
chunk_fwd_segmented(q, k, v, beta, lam, log_alpha=None, initial_state=None, n_segments=None,
          save_states=False) -> (o, final_state, saved)   (dense; long sequences, few heads)
chunk_bwd(q, k, v, beta, lam, log_alpha, initial_state, saved_states, d_o,
          d_final_state=None, cu_seqlens=None) -> dict of gradients
recurrent_step(q, k, v, beta, lam, log_alpha, state) -> o        (state updated in place)
recurrent_fwd(q, k, v, beta, lam=None, log_alpha=None, initial_state=None, cu_seqlens=None)
          -> (o, final_state)                                  (token by token, one launch)
recurrent_bwd(q, k, v, beta, lam, log_alpha, initial_state, d_o, d_final_state=None,
          cu_seqlens=None) -> dict of gradients                (token by token, one launch)
l2norm_fwd(x) -> (y, rnorm);  l2norm_bwd(y, rnorm, dy) -> dx   (row L2 norm for the layer's q, k)

lam: a [.., H] fp32 tensor (per token and head), a number (one constant for every
token and head: the paper's fixed-lambda ablations), or None (lambda == 0, the gated
delta rule); log_alpha=None means alpha == 1.
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libqdelta.so")
CHUNK = 64

QDELTA_OK, QDELTA_EINVAL, QDELTA_EUNSUPPORTED, QDELTA_ENOWORKSPACE, QDELTA_EHIP = range(5)
QDELTA_F32, QDELTA_BF16 = 0, 1

EXPORTS = (
    "qdelta_status_string", "qdelta_version", "qdelta_saved_state_slots", "qdelta_saved_bytes",
    "qdelta_chunk_workspace_bytes", "qdelta_chunk_fwd", "qdelta_chunk_fwd_varlen",
    "qdelta_chunk_bwd", "qdelta_chunk_bwd_varlen", "qdelta_recurrent_step",
    "qdelta_recurrent_fwd", "qdelta_recurrent_fwd_varlen", "qdelta_l2norm_fwd", "qdelta_l2norm_bwd",
    "qdelta_profile_begin", "qdelta_profile_end", "qdelta_chunk_fwd_noalloc",
    "qdelta_chunk_fwd_segmented", "qdelta_segmented_workspace_bytes", "qdelta_suggest_segments",
    "qdelta_recurrent_workspace_bytes", "qdelta_recurrent_bwd", "qdelta_recurrent_bwd_varlen",
)
NOALLOC_SCRATCH_BYTES = 64 << 20

STAGES = ("prep_fwd", "scan_fwd", "prep_bwd", "scan_bwd", "intra", "step", "rec_fwd", "seg_maps",
          "seg_compose", "seg_out", "rec_bwd")

_lib = None


class QDeltaError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        msg = lib().qdelta_status_string(status).decode() if _lib is not None else str(status)
        super().__init__(f"{fn} failed with status {status}: {msg}")


def lib():
    """Load libqdelta.so (raises if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run paper_2606_08804_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        i32, sz, P = ctypes.c_int32, ctypes.c_size_t, ctypes.c_void_p
        L.qdelta_status_string.argtypes = [ctypes.c_int]
        L.qdelta_status_string.restype = ctypes.c_char_p
        L.qdelta_version.argtypes = []
        L.qdelta_version.restype = ctypes.c_int
        L.qdelta_saved_state_slots.argtypes = [i32, i32, i32, i32]
        L.qdelta_saved_state_slots.restype = sz
        L.qdelta_saved_bytes.argtypes = [i32] * 8
        L.qdelta_saved_bytes.restype = sz
        L.qdelta_chunk_workspace_bytes.argtypes = [i32] * 9
        L.qdelta_chunk_workspace_bytes.restype = sz
        f32 = ctypes.c_float
        # gate arguments: beta, lam, lam_scalar, log_alpha
        L.qdelta_chunk_fwd.argtypes = [i32] * 7 + [P] * 5 + [f32] + [P] * 5 + [P, sz, P]
        L.qdelta_chunk_fwd.restype = ctypes.c_int
        L.qdelta_chunk_fwd_noalloc.argtypes = [i32] * 7 + [P] * 5 + [f32] + [P] * 4 + [P]
        L.qdelta_chunk_fwd_noalloc.restype = ctypes.c_int
        L.qdelta_chunk_fwd_segmented.argtypes = [i32] * 7 + [P] * 5 + [f32] + [P] * 5 + [i32, P, sz, P]
        L.qdelta_chunk_fwd_segmented.restype = ctypes.c_int
        L.qdelta_segmented_workspace_bytes.argtypes = [i32] * 8
        L.qdelta_segmented_workspace_bytes.restype = sz
        L.qdelta_suggest_segments.argtypes = [i32] * 6
        L.qdelta_suggest_segments.restype = i32
        L.qdelta_chunk_fwd_varlen.argtypes = [i32, i32, P] + [i32] * 5 + [P] * 5 + [f32] + [P] * 5 + [P, sz, P]
        L.qdelta_chunk_fwd_varlen.restype = ctypes.c_int
        L.qdelta_chunk_bwd.argtypes = [i32] * 7 + [P] * 5 + [f32] + [P] * 12 + [P, sz, P]
        L.qdelta_chunk_bwd.restype = ctypes.c_int
        L.qdelta_chunk_bwd_varlen.argtypes = [i32, i32, P] + [i32] * 5 + [P] * 5 + [f32] + [P] * 12 + [P, sz, P]
        L.qdelta_chunk_bwd_varlen.restype = ctypes.c_int
        L.qdelta_recurrent_step.argtypes = [i32] * 5 + [P] * 5 + [f32] + [P] * 3 + [P]
        L.qdelta_recurrent_step.restype = ctypes.c_int
        L.qdelta_recurrent_fwd.argtypes = [i32] * 6 + [P] * 5 + [f32] + [P] * 4 + [P]
        L.qdelta_recurrent_fwd.restype = ctypes.c_int
        L.qdelta_recurrent_fwd_varlen.argtypes = [i32, i32, P] + [i32] * 4 + [P] * 5 + [f32] + [P] * 4 + [P]
        L.qdelta_recurrent_fwd_varlen.restype = ctypes.c_int
        L.qdelta_recurrent_workspace_bytes.argtypes = [i32] * 6
        L.qdelta_recurrent_workspace_bytes.restype = sz
        # q, k, v, beta, lam, lam_scalar, log_alpha, S0, dO, dSf, dq, dk, dv, dbeta, dlam, dla, dS0, ws, bytes, stream
        L.qdelta_recurrent_bwd.argtypes = [i32] * 6 + [P] * 5 + [f32] + [P] * 11 + [P, sz, P]
        L.qdelta_recurrent_bwd.restype = ctypes.c_int
        L.qdelta_recurrent_bwd_varlen.argtypes = [i32, i32, P] + [i32] * 4 + [P] * 5 + [f32] + [P] * 11 + [P, sz, P]
        L.qdelta_recurrent_bwd_varlen.restype = ctypes.c_int
        i64 = ctypes.c_int64
        L.qdelta_l2norm_fwd.argtypes = [i64, i32, i64, i32, P, P, P, P]
        L.qdelta_l2norm_fwd.restype = ctypes.c_int
        L.qdelta_l2norm_bwd.argtypes = [i64, i32, i32, P, P, P, P, P]
        L.qdelta_l2norm_bwd.restype = ctypes.c_int
        L.qdelta_profile_begin.argtypes = []
        L.qdelta_profile_begin.restype = ctypes.c_int
        L.qdelta_profile_end.argtypes = [P, P]
        L.qdelta_profile_end.restype = ctypes.c_int
        _lib = L
    return _lib


def _dt(t):
    if t.dtype == torch.bfloat16:
        return QDELTA_BF16
    if t.dtype == torch.float32:
        return QDELTA_F32
    raise TypeError(f"unsupported activation dtype {t.dtype}")


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _need(t, name, dtype=None, shape=None):
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def _opt(t, name, dtype=None, shape=None):
    return None if t is None else _need(t, name, dtype, shape)


def _lam(lam, shape):
    """lambda as (tensor or None, constant): a tensor is per token and head;
    None or a number is one constant for every token and head (None = 0,
    the gated delta rule)."""
    if lam is None:
        return None, 0.0
    if isinstance(lam, (int, float)):
        return None, float(lam)
    return _need(lam, "lam", torch.float32, shape), 0.0


def _check(fn, status):
    if status != QDELTA_OK:
        raise QDeltaError(fn, status)


def _dims(q, v, cu_seqlens):
    if cu_seqlens is None:
        B, T, H, Dk = q.shape
        N = B
    else:
        if q.dim() == 4:
            if q.shape[0] != 1:
                raise ValueError("a packed batch has leading dimension 1")
            _, T, H, Dk = q.shape
        else:
            T, H, Dk = q.shape
        B = 1
        N = cu_seqlens.numel() - 1
    return B, T, H, Dk, v.shape[-1], N


def saved_state_slots(B, T, n_seqs=0):
    return int(lib().qdelta_saved_state_slots(B, T, CHUNK, n_seqs))


def saved_bytes(B, T, H, Dk, Dv, dtype, n_seqs=0):
    """Bytes of the saved context (per-chunk states and new values) for the backward."""
    return int(lib().qdelta_saved_bytes(B, T, H, Dk, Dv, CHUNK, dtype, n_seqs))


def workspace_bytes(B, T, H, Dk, Dv, dtype, n_seqs=0, is_bwd=False):
    return int(lib().qdelta_chunk_workspace_bytes(B, T, H, Dk, Dv, CHUNK, dtype, n_seqs, int(is_bwd)))


def _workspace(nbytes, device, workspace):
    if nbytes == 0:
        return None
    if workspace is not None:
        if workspace.numel() * workspace.element_size() < nbytes:
            raise ValueError("workspace too small")
        return workspace
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def chunk_fwd(q, k, v, beta, lam, log_alpha=None, initial_state=None, cu_seqlens=None,
              output_final_state=True, save_states=False, workspace=None):
    """Chunkwise Q-Delta forward.  Returns (o, final_state or None, saved_states or None)."""
    L = lib()
    dt = _dt(q)
    B, T, H, Dk, Dv, N = _dims(q, v, cu_seqlens)
    act = q.shape[:-1]
    _need(q, "q", q.dtype)
    _need(k, "k", q.dtype, q.shape)
    _need(v, "v", q.dtype, tuple(act) + (Dv,))
    _need(beta, "beta", torch.float32, act)
    lam_t, lam_c = _lam(lam, act)
    _opt(log_alpha, "log_alpha", torch.float32, act)
    _opt(initial_state, "initial_state", torch.float32, (N, H, Dv, Dk))
    if cu_seqlens is not None:
        _need(cu_seqlens, "cu_seqlens", torch.int32)
    dev = q.device
    o = torch.empty(tuple(act) + (Dv,), dtype=q.dtype, device=dev)
    Sf = torch.empty((N, H, Dv, Dk), dtype=torch.float32, device=dev) if output_final_state else None
    n_seqs = N if cu_seqlens is not None else 0
    saved = None
    if save_states:
        saved = torch.empty(saved_bytes(B, T, H, Dk, Dv, dt, n_seqs), dtype=torch.uint8, device=dev)
    nbytes = workspace_bytes(B, T, H, Dk, Dv, dt, n_seqs, False)
    ws = _workspace(nbytes, dev, workspace)
    common = (H, Dk, Dv, CHUNK, dt, _p(q), _p(k), _p(v), _p(beta), _p(lam_t), lam_c, _p(log_alpha),
              _p(initial_state), _p(o), _p(Sf), _p(saved), _p(ws), nbytes, _stream())
    if cu_seqlens is None:
        _check("qdelta_chunk_fwd", L.qdelta_chunk_fwd(B, T, *common))
    else:
        _check("qdelta_chunk_fwd_varlen", L.qdelta_chunk_fwd_varlen(T, N, _p(cu_seqlens), *common))
    return o, Sf, saved


def suggest_segments(B, T, H, Dk, Dv, dtype=QDELTA_BF16):
    """Segment count the segment-parallel forward is expected to run fastest
    with on the current device (1: the single pass)."""
    return int(lib().qdelta_suggest_segments(B, T, H, Dk, Dv, dtype))


def segmented_workspace_bytes(B, T, H, Dk, Dv, dtype, n_segments):
    return int(lib().qdelta_segmented_workspace_bytes(B, T, H, Dk, Dv, CHUNK, dtype, n_segments))


def chunk_fwd_segmented(q, k, v, beta, lam, log_alpha=None, initial_state=None, n_segments=None,
                        output_final_state=True, save_states=False, workspace=None):
    """Segment-parallel chunkwise forward of a dense batch (long sequences,
    few (sequence, head) pairs).  n_segments None: the library's suggestion
    for this device.  Returns (o, final_state or None, saved or None), as
    chunk_fwd."""
    L = lib()
    dt = _dt(q)
    B, T, H, Dk, Dv, N = _dims(q, v, None)
    act = q.shape[:-1]
    _need(q, "q", q.dtype)
    _need(k, "k", q.dtype, q.shape)
    _need(v, "v", q.dtype, tuple(act) + (Dv,))
    _need(beta, "beta", torch.float32, act)
    lam_t, lam_c = _lam(lam, act)
    _opt(log_alpha, "log_alpha", torch.float32, act)
    _opt(initial_state, "initial_state", torch.float32, (N, H, Dv, Dk))
    G = suggest_segments(B, T, H, Dk, Dv, dt) if n_segments is None else int(n_segments)
    dev = q.device
    o = torch.empty(tuple(act) + (Dv,), dtype=q.dtype, device=dev)
    Sf = torch.empty((N, H, Dv, Dk), dtype=torch.float32, device=dev) if output_final_state else None
    saved = None
    if save_states:
        saved = torch.empty(saved_bytes(B, T, H, Dk, Dv, dt, 0), dtype=torch.uint8, device=dev)
    nbytes = segmented_workspace_bytes(B, T, H, Dk, Dv, dt, max(G, 1))
    ws = _workspace(nbytes, dev, workspace)
    _check("qdelta_chunk_fwd_segmented",
           L.qdelta_chunk_fwd_segmented(B, T, H, Dk, Dv, CHUNK, dt, _p(q), _p(k), _p(v), _p(beta), _p(lam_t),
                                        lam_c, _p(log_alpha), _p(initial_state), _p(o), _p(Sf), _p(saved), G,
                                        _p(ws), nbytes, _stream()))
    return o, Sf, saved


def chunk_fwd_noalloc(q, k, v, beta, lam, log_alpha=None, initial_state=None, out=None,
                      final_state_out=None, output_final_state=True):
    """Dense chunkwise forward through qdelta_chunk_fwd_noalloc: no workspace
    and no saved context; the library uses its own per-device scratch array.
    Outputs may be passed in (out [B,T,H,Dv], final_state_out [B,H,Dv,Dk]) so
    that this call allocates nothing either.  Returns (o, final_state or None)."""
    L = lib()
    dt = _dt(q)
    B, T, H, Dk, Dv, N = _dims(q, v, None)
    act = q.shape[:-1]
    _need(q, "q", q.dtype)
    _need(k, "k", q.dtype, q.shape)
    _need(v, "v", q.dtype, tuple(act) + (Dv,))
    _need(beta, "beta", torch.float32, act)
    lam_t, lam_c = _lam(lam, act)
    _opt(log_alpha, "log_alpha", torch.float32, act)
    _opt(initial_state, "initial_state", torch.float32, (N, H, Dv, Dk))
    o = out if out is not None else torch.empty(tuple(act) + (Dv,), dtype=q.dtype, device=q.device)
    _need(o, "out", q.dtype, tuple(act) + (Dv,))
    Sf = final_state_out
    if Sf is None and output_final_state:
        Sf = torch.empty((N, H, Dv, Dk), dtype=torch.float32, device=q.device)
    _opt(Sf, "final_state_out", torch.float32, (N, H, Dv, Dk))
    _check("qdelta_chunk_fwd_noalloc",
           L.qdelta_chunk_fwd_noalloc(B, T, H, Dk, Dv, CHUNK, dt, _p(q), _p(k), _p(v), _p(beta), _p(lam_t),
                                      lam_c, _p(log_alpha), _p(initial_state), _p(o), _p(Sf), _stream()))
    return o, Sf


def chunk_bwd(q, k, v, beta, lam, log_alpha, initial_state, saved_states, d_o,
              d_final_state=None, cu_seqlens=None, need_d_initial_state=True, workspace=None):
    """Chunkwise Q-Delta backward.  Returns a dict: dq, dk, dv, dbeta, dlam
    (per token for a lam tensor; a 0-dim tensor, the gradient of the
    constant, when lam is a number; None when lam is None), dlog_alpha (None
    without decay), d_initial_state (None if not requested)."""
    L = lib()
    dt = _dt(q)
    B, T, H, Dk, Dv, N = _dims(q, v, cu_seqlens)
    act = q.shape[:-1]
    _need(q, "q", q.dtype)
    _need(k, "k", q.dtype, q.shape)
    _need(v, "v", q.dtype, tuple(act) + (Dv,))
    _need(beta, "beta", torch.float32, act)
    lam_t, lam_c = _lam(lam, act)
    _opt(log_alpha, "log_alpha", torch.float32, act)
    _opt(initial_state, "initial_state", torch.float32, (N, H, Dv, Dk))
    _opt(saved_states, "saved_states")
    _need(d_o, "d_o", q.dtype, tuple(act) + (Dv,))
    _opt(d_final_state, "d_final_state", torch.float32, (N, H, Dv, Dk))
    if cu_seqlens is not None:
        _need(cu_seqlens, "cu_seqlens", torch.int32)
    n_seqs = N if cu_seqlens is not None else 0
    if saved_states is not None:
        nb = saved_bytes(B, T, H, Dk, Dv, dt, n_seqs)
        if saved_states.dtype != torch.uint8 or saved_states.numel() < nb:
            raise ValueError(f"saved_states must be a uint8 buffer of at least {nb} bytes")
    dev = q.device
    dq = torch.empty_like(q)
    dk = torch.empty_like(k)
    dv = torch.empty_like(v)
    dbeta = torch.empty_like(beta)
    if lam_t is not None:
        dlam = torch.empty_like(lam_t)
    elif lam is not None:
        dlam = torch.empty((), dtype=torch.float32, device=dev)
    else:
        dlam = None
    dla = torch.empty_like(log_alpha) if log_alpha is not None else None
    dS0 = torch.empty((N, H, Dv, Dk), dtype=torch.float32, device=dev) if need_d_initial_state else None
    nbytes = workspace_bytes(B, T, H, Dk, Dv, dt, n_seqs, True)
    ws = _workspace(nbytes, dev, workspace)
    common = (H, Dk, Dv, CHUNK, dt, _p(q), _p(k), _p(v), _p(beta), _p(lam_t), lam_c, _p(log_alpha),
              _p(initial_state), _p(saved_states), _p(d_o), _p(d_final_state), _p(dq), _p(dk),
              _p(dv), _p(dbeta), _p(dlam), _p(dla), _p(dS0), _p(ws), nbytes, _stream())
    if cu_seqlens is None:
        _check("qdelta_chunk_bwd", L.qdelta_chunk_bwd(B, T, *common))
    else:
        _check("qdelta_chunk_bwd_varlen", L.qdelta_chunk_bwd_varlen(T, N, _p(cu_seqlens), *common))
    return dict(dq=dq, dk=dk, dv=dv, dbeta=dbeta, dlam=dlam, dlog_alpha=dla, d_initial_state=dS0)


def recurrent_step(q, k, v, beta, lam, log_alpha, state, out=None):
    """One token for N sequences: q,k [N,H,Dk], v [N,H,Dv], gates [N,H],
    state [N,H,Dv,Dk] fp32 (updated in place).  Returns o [N,H,Dv]."""
    L = lib()
    dt = _dt(q)
    N, H, Dk = q.shape
    Dv = v.shape[-1]
    _need(q, "q", q.dtype)
    _need(k, "k", q.dtype, q.shape)
    _need(v, "v", q.dtype, (N, H, Dv))
    _need(beta, "beta", torch.float32, (N, H))
    lam_t, lam_c = _lam(lam, (N, H))
    _opt(log_alpha, "log_alpha", torch.float32, (N, H))
    _need(state, "state", torch.float32, (N, H, Dv, Dk))
    o = out if out is not None else torch.empty((N, H, Dv), dtype=q.dtype, device=q.device)
    _need(o, "out", q.dtype, (N, H, Dv))
    _check("qdelta_recurrent_step",
           L.qdelta_recurrent_step(N, H, Dk, Dv, dt, _p(q), _p(k), _p(v), _p(beta), _p(lam_t), lam_c,
                                   _p(log_alpha), _p(state), _p(o), _stream()))
    return o


def recurrent_fwd(q, k, v, beta, lam=None, log_alpha=None, initial_state=None, cu_seqlens=None,
                  output_final_state=True):
    """Fully recurrent forward (token by token, one launch).  Same layouts as
    chunk_fwd.  Returns (o, final_state or None)."""
    L = lib()
    dt = _dt(q)
    B, T, H, Dk, Dv, N = _dims(q, v, cu_seqlens)
    act = q.shape[:-1]
    _need(q, "q", q.dtype)
    _need(k, "k", q.dtype, q.shape)
    _need(v, "v", q.dtype, tuple(act) + (Dv,))
    _need(beta, "beta", torch.float32, act)
    lam_t, lam_c = _lam(lam, act)
    _opt(log_alpha, "log_alpha", torch.float32, act)
    _opt(initial_state, "initial_state", torch.float32, (N, H, Dv, Dk))
    if cu_seqlens is not None:
        _need(cu_seqlens, "cu_seqlens", torch.int32)
    o = torch.empty(tuple(act) + (Dv,), dtype=q.dtype, device=q.device)
    Sf = torch.empty((N, H, Dv, Dk), dtype=torch.float32, device=q.device) if output_final_state else None
    common = (H, Dk, Dv, dt, _p(q), _p(k), _p(v), _p(beta), _p(lam_t), lam_c, _p(log_alpha),
              _p(initial_state), _p(o), _p(Sf), _stream())
    if cu_seqlens is None:
        _check("qdelta_recurrent_fwd", L.qdelta_recurrent_fwd(B, T, *common))
    else:
        _check("qdelta_recurrent_fwd_varlen",
               L.qdelta_recurrent_fwd_varlen(T, N, _p(cu_seqlens), *common))
    return o, Sf


def recurrent_workspace_bytes(B, T, H, Dk, Dv, n_seqs=0):
    return int(lib().qdelta_recurrent_workspace_bytes(B, T, H, Dk, Dv, n_seqs))


def recurrent_bwd(q, k, v, beta, lam, log_alpha, initial_state, d_o, d_final_state=None, cu_seqlens=None,
                  need_d_initial_state=True, workspace=None):
    """Backward of the fully recurrent form (token by token, one launch, no
    saved context).  Same layouts and returned gradients as chunk_bwd."""
    L = lib()
    dt = _dt(q)
    B, T, H, Dk, Dv, N = _dims(q, v, cu_seqlens)
    act = q.shape[:-1]
    _need(q, "q", q.dtype)
    _need(k, "k", q.dtype, q.shape)
    _need(v, "v", q.dtype, tuple(act) + (Dv,))
    _need(beta, "beta", torch.float32, act)
    lam_t, lam_c = _lam(lam, act)
    _opt(log_alpha, "log_alpha", torch.float32, act)
    _opt(initial_state, "initial_state", torch.float32, (N, H, Dv, Dk))
    _need(d_o, "d_o", q.dtype, tuple(act) + (Dv,))
    _opt(d_final_state, "d_final_state", torch.float32, (N, H, Dv, Dk))
    if cu_seqlens is not None:
        _need(cu_seqlens, "cu_seqlens", torch.int32)
    dev = q.device
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    dbeta = torch.empty_like(beta)
    if lam_t is not None:
        dlam = torch.empty_like(lam_t)
    elif lam is not None:
        dlam = torch.empty((), dtype=torch.float32, device=dev)
    else:
        dlam = None
    dla = torch.empty_like(log_alpha) if log_alpha is not None else None
    dS0 = torch.empty((N, H, Dv, Dk), dtype=torch.float32, device=dev) if need_d_initial_state else None
    n_seqs = N if cu_seqlens is not None else 0
    nbytes = recurrent_workspace_bytes(B, T, H, Dk, Dv, n_seqs)
    ws = _workspace(nbytes, dev, workspace)
    common = (H, Dk, Dv, dt, _p(q), _p(k), _p(v), _p(beta), _p(lam_t), lam_c, _p(log_alpha), _p(initial_state),
              _p(d_o), _p(d_final_state), _p(dq), _p(dk), _p(dv), _p(dbeta), _p(dlam), _p(dla), _p(dS0),
              _p(ws), nbytes, _stream())
    if cu_seqlens is None:
        _check("qdelta_recurrent_bwd", L.qdelta_recurrent_bwd(B, T, *common))
    else:
        _check("qdelta_recurrent_bwd_varlen", L.qdelta_recurrent_bwd_varlen(T, N, _p(cu_seqlens), *common))
    return dict(dq=dq, dk=dk, dv=dv, dbeta=dbeta, dlam=dlam, dlog_alpha=dla, d_initial_state=dS0)


def l2norm_fwd(x):
    """Row L2 normalisation over the last dim of x (rows may be strided, as in a
    slice of a fused projection).  Returns (y contiguous, rnorm [rows] fp32)."""
    D = x.shape[-1]
    if not x.is_cuda:
        raise ValueError("x must be a device tensor")
    ld = x.stride(-2) if x.dim() >= 2 else D
    expected = ld
    for i in range(x.dim() - 3, -1, -1):    # leading dims must collapse into one row index
        expected *= x.shape[i + 1]
        if x.shape[i] > 1 and x.stride(i) != expected:
            raise ValueError("x must have evenly strided rows")
    if x.stride(-1) != 1:
        raise ValueError("x must have unit stride in its last dim")
    y = torch.empty(x.shape, dtype=x.dtype, device=x.device)
    rn = torch.empty(x.shape[:-1], dtype=torch.float32, device=x.device)
    _check("qdelta_l2norm_fwd", lib().qdelta_l2norm_fwd(x.numel() // D, D, ld, _dt(x), _p(x), _p(y),
                                                        _p(rn), _stream()))
    return y, rn


def l2norm_bwd(y, rn, dy):
    """dx for l2norm_fwd (contiguous, shaped like y)."""
    _need(y, "y", y.dtype)
    _need(dy, "dy", y.dtype, tuple(y.shape))
    _need(rn, "rnorm", torch.float32, tuple(y.shape[:-1]))
    dx = torch.empty_like(y)
    _check("qdelta_l2norm_bwd", lib().qdelta_l2norm_bwd(y.numel() // y.shape[-1], y.shape[-1], _dt(y),
                                                        _p(y), _p(rn), _p(dy), _p(dx), _stream()))
    return dx


def profile_begin():
    """Start timing every library kernel launch with HIP events (per stage)."""
    _check("qdelta_profile_begin", lib().qdelta_profile_begin())


def profile_end():
    """Stop timing; returns {stage: (total_ms, launches)}."""
    n = len(STAGES)
    ms = (ctypes.c_float * n)()
    cnt = (ctypes.c_int32 * n)()
    _check("qdelta_profile_end", lib().qdelta_profile_end(ms, cnt))
    return {name: (float(ms[i]), int(cnt[i])) for i, name in enumerate(STAGES)}
