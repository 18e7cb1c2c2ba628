"""The saved context that the forward writes for the backward, decoded on the
host by its documented layout (entry states, D in 32-value-column tiles, the
gate block, a zero block, P and M as their ten 16 x 16 blocks on and below the
diagonal, one region after the other) and compared region by region with the
fp64 chunk algebra of the oracle (Sec. 3.3 chunkwise form; App. D.1 and D.2):
per chunk the entry state S, D = U - W S^T, the chunk-local prefix sums b with
beta and lambda, P = Gam * M_causal * Q K^T and (I + A)^{-1}, whose blocks
above the diagonal the oracle's own values show to be zero.

What the layout promises beyond the values is checked exactly: rows of D and P
past a chunk's end are zero, so are beta and lambda there and the zero
block.  The cases cover a ragged last chunk, packed sequences with slot holes,
and a shape whose scan writes two D tiles per workgroup (64 value rows per
workgroup) and whose backward scan takes zero rows from the zero block.

Tolerances: normwise max error per region over the whole batch, 1e-4 for fp32
inputs and 2e-2 for bf16 (the regions are stored in the activation dtype;
the gate block is fp32 in both)."""
import numpy as np
import pytest
import torch

from oracle import chunk
from paper_2606_08804_amd import qdelta, synth
from tests.gpu_helpers import TOL, bwd_errors, f64, gpu_bwd, gpu_fwd, normwise

pytestmark = pytest.mark.gpu

C = 64


def _unpack(blocks):
    """[units, 10, 16, 16] lower 16 x 16 blocks -> [units, C, C] (zeros above)."""
    out = np.zeros((blocks.shape[0], C, C))
    for r in range(4):
        for c in range(r + 1):
            out[:, 16 * r:16 * r + 16, 16 * c:16 * c + 16] = blocks[:, r * (r + 1) // 2 + c]
    return out


def _regions(saved, units, Dk, Dv, dt):
    """Split the context bytes into its six regions, as float64 arrays."""
    e = 2 if dt == "bf16" else 4
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    raw = saved.cpu()
    sizes = [units * Dv * Dk * e, units * C * Dv * e, units * 3 * C * 4, 1024, units * 2560 * e, units * 2560 * e]
    assert sum(sizes) == raw.numel()
    out, off = [], 0
    for i, n in enumerate(sizes):
        b = raw[off:off + n]
        off += n
        out.append(b.numpy().astype(np.float64) if i == 3 else
                   b.view(torch.float32 if i == 2 else tdt).to(torch.float64).numpy())
    S, D, G, Z, P, M = out
    assert not Z.any(), "zero block"
    return (S.reshape(units, Dv, Dk), D.reshape(units, Dv // 32, C, 32), G.reshape(units, 3, C),
            _unpack(P.reshape(units, 10, 16, 16)), _unpack(M.reshape(units, 10, 16, 16)))


def _sequences(d):
    """(sequence index, token slice into the packed or dense batch, first slot)."""
    cu = d["cu_seqlens"]
    if cu is None:
        B, T = d["q"].shape[:2]
        nt = (T + C - 1) // C
        return [(n, n, slice(0, T), n * nt) for n in range(B)]
    cu = cu.tolist()
    return [(n, 0, slice(cu[n], cu[n + 1]), cu[n] // C + n) for n in range(len(cu) - 1)]


def _pad(x):
    """Rows of a chunk operator widened to C columns with zeros."""
    out = np.zeros((x.shape[0], C))
    out[:, :x.shape[1]] = x
    return out


def _check_context(d, dt):
    B, T, H, Dk = d["q"].shape
    Dv = d["v"].shape[3]
    n_seqs = 0 if d["cu_seqlens"] is None else len(d["cu_seqlens"]) - 1
    _, _, saved = gpu_fwd(d, save_states=True)
    units = qdelta.saved_state_slots(B, T, n_seqs) * H
    S, D, G, P, M = _regions(saved, units, Dk, Dv, dt)
    got = {k: [] for k in ("S", "D", "b", "beta", "lam", "P", "M")}
    ref = {k: [] for k in got}
    for n, bi, sl, slot0 in _sequences(d):
        for h in range(H):
            q = f64(d["q"][bi, sl, h])
            k = f64(d["k"][bi, sl, h])
            v = f64(d["v"][bi, sl, h])
            be = f64(d["beta"][bi, sl, h])
            lm = f64(d["lam"][bi, sl, h])
            la = np.zeros(q.shape[0]) if d["log_alpha"] is None else f64(d["log_alpha"][bi, sl, h])
            S0 = np.zeros((Dv, Dk)) if d["initial_state"] is None else f64(d["initial_state"][n, h])
            _, _, states = chunk.fwd_unit(q, k, v, be, lm, la, S0, C)
            for c, Sc in enumerate(states):
                cs = slice(c * C, min((c + 1) * C, q.shape[0]))
                ln = cs.stop - cs.start
                st = chunk._chunk_setup(q[cs], k[cs], v[cs], be[cs], lm[cs], la[cs])
                u = (slot0 + c) * H + h
                Dfull = np.concatenate(list(D[u]), axis=1)          # tiles side by side: C x Dv
                assert not Dfull[ln:].any(), f"D rows past the chunk (seq {n} head {h} chunk {c})"
                assert not P[u, ln:].any(), f"P rows past the chunk (seq {n} head {h} chunk {c})"
                assert not G[u, 1, ln:].any() and not G[u, 2, ln:].any(), "beta, lambda past the chunk"
                for key, g_, r_ in (("S", S[u], Sc), ("D", Dfull[:ln], st["U"] - st["W"] @ Sc.T),
                                    ("b", G[u, 0, :ln], st["b"]), ("beta", G[u, 1, :ln], be[cs]),
                                    ("lam", G[u, 2, :ln], lm[cs]), ("P", P[u, :ln], _pad(st["Pm"])),
                                    ("M", M[u, :ln, :ln], st["Minv"])):
                    got[key].append(np.ravel(g_))
                    ref[key].append(np.ravel(r_))
    errs = {key: normwise(np.concatenate(got[key]), np.concatenate(ref[key])) for key in got}
    tol = {key: TOL["f32"] if key in ("b", "beta", "lam") else TOL[dt] for key in errs}
    bad = {key: e for key, e in errs.items() if not e <= tol[key]}
    assert not bad, f"context regions off: {errs}"
    return errs


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_context_dense_ragged(dt):
    """Two sequences of 150 tokens (chunks of 64, 64 and 22), two D tiles."""
    d = synth.make(2, 150, 2, 64, 64, dt, "G2", seed=131, s0=True)
    _check_context(d, dt)


def test_context_bf16_d128():
    """Head dims of the training shape (Dk = Dv = 128, four D tiles)."""
    d = synth.make(1, 100, 2, 128, 128, "bf16", "G3", seed=132, s0=True)
    _check_context(d, "bf16")


def test_context_varlen_holes():
    """Packed sequences of 70, 5 and 130 tokens: slot holes between them."""
    d = synth.make(1, 0, 2, 64, 128, "bf16", "G2", seed=133, s0=True, lengths=[70, 5, 130])
    _check_context(d, "bf16")


def test_context_wide_scan_tiles_and_backward():
    """512 (sequence, head) pairs of 70 tokens: the scans run 64 value rows
    per workgroup, so each forward workgroup writes two D tiles and the
    backward scan takes the zero rows of its output-gradient tiles (last
    chunk of 6 tokens) from the zero block; the backward is checked against
    the oracle."""
    d = synth.make(32, 70, 16, 64, 128, "bf16", "G2", seed=134, s0=True, with_do=True)
    _check_context(d, "bf16")
    errs = bwd_errors(d, gpu_bwd(d))
    assert all(e <= TOL["bf16"] for e in errs.values()), errs
