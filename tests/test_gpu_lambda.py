"""The constant-lambda form of every entry point (lam == NULL with a scalar,
the paper's fixed-lambda ablations: 0.2, 0.5, 0.8 and 1, Sec. 4.2) against
the fp64 oracle run with that constant at every token and head, and against
the library's own per-token path given a filled lambda tensor: the forward
results are the same bit for bit (the kernels read the same value), the
gradients agree, and the constant's gradient is the sum of the per-token
lambda gradients."""
import numpy as np
import pytest
import torch

from paper_2606_08804_amd import qdelta, synth
from tests.gpu_helpers import TOL, bwd_errors, dev, f64, fwd_errors, normwise, oracle_bwd, oracle_fwd

pytestmark = pytest.mark.gpu

LAMBDAS = [0.2, 0.5, 0.8, 1.0]


def _filled(d, c):
    return dict(d, lam=torch.full_like(d["beta"], c))


def _fwd(d, lam):
    o, Sf, saved = qdelta.chunk_fwd(dev(d["q"]), dev(d["k"]), dev(d["v"]), dev(d["beta"]), lam,
                                    dev(d["log_alpha"]), dev(d["initial_state"]),
                                    cu_seqlens=dev(d["cu_seqlens"]), save_states=True)
    torch.cuda.synchronize()
    return o, Sf, saved


def _bwd(d, lam, saved):
    g = qdelta.chunk_bwd(dev(d["q"]), dev(d["k"]), dev(d["v"]), dev(d["beta"]), lam, dev(d["log_alpha"]),
                         dev(d["initial_state"]), saved, dev(d["d_o"]), cu_seqlens=dev(d["cu_seqlens"]))
    torch.cuda.synchronize()
    return g


@pytest.mark.parametrize("c", LAMBDAS)
@pytest.mark.parametrize("dt,varlen", [("bf16", False), ("f32", False), ("bf16", True)])
def test_chunk_constant_lambda(c, dt, varlen):
    D = 128 if dt == "bf16" else 64
    gate = "G3" if varlen else "G2"
    if varlen:
        d = synth.make(1, 0, 2, D, D, dt, gate, seed=160, s0=True, with_do=True, lengths=[70, 1, 130, 64])
    else:
        d = synth.make(2, 150, 2, D, D, dt, gate, seed=161, s0=True, with_do=True)
    dc = _filled(d, c)
    tol = TOL[dt]
    o, Sf, saved = _fwd(d, c)
    e = fwd_errors(dc, o, Sf)
    assert all(v <= tol for v in e.values()), e
    # the filled-tensor path reads the same lambda values: identical forward
    o_t, Sf_t, saved_t = _fwd(dc, dev(dc["lam"]))
    assert torch.equal(o, o_t) and torch.equal(Sf, Sf_t)
    if not varlen:
        # (a packed batch leaves the context slots no chunk maps to untouched)
        assert torch.equal(saved, saved_t)

    g = _bwd(d, c, saved)
    assert g["dlam"].shape == ()
    e = bwd_errors(dc, g, skip=("dlam",))
    assert all(v <= tol for v in e.values()), e
    ref = oracle_bwd(dc)["dlam"]
    got = float(g["dlam"].cpu())
    # a sum over every (token, head) with cancellation: error against the
    # sum of the summands' magnitudes
    assert abs(got - ref.sum()) <= tol * np.abs(ref).sum(), (got, ref.sum())
    # the per-token path on the filled tensor: equal gradients, and the
    # constant's gradient equals the sum of its per-token gradients
    g_t = _bwd(dc, dev(dc["lam"]), saved_t)
    for key in ("dq", "dk", "dv", "dbeta", "dlog_alpha", "d_initial_state"):
        if g[key] is not None:
            assert torch.equal(g[key], g_t[key]), key
    per_token = f64(g_t["dlam"].cpu())
    assert abs(got - per_token.sum()) <= 1e-5 * np.abs(per_token).sum() + 1e-30


def test_chunk_constant_lambda_no_gradient_and_empty():
    """lam = a number with no sequences: the constant's gradient is written
    as zero; lam = None still means the gated delta rule with no dlam."""
    d = synth.make(0, 64, 2, 64, 64, "bf16", "G2", seed=162, s0=False, with_do=True)
    q = dev(d["q"])
    g = qdelta.chunk_bwd(q, dev(d["k"]), dev(d["v"]), dev(d["beta"]), 0.5, dev(d["log_alpha"]), None, None,
                         dev(d["d_o"]))
    torch.cuda.synchronize()
    assert float(g["dlam"].cpu()) == 0.0


@pytest.mark.parametrize("c", LAMBDAS)
def test_recurrent_step_constant_lambda(c):
    N, H, D = 8, 4, 128
    d = synth.make(1, N, H, D, D, "bf16", "G2", seed=163)
    S = torch.from_numpy(np.random.default_rng(7).normal(0, 0.02, (N, H, D, D)).astype(np.float32))
    Sa, Sb = S.cuda(), S.cuda()
    args = [d[key][0].cuda() for key in ("q", "k", "v", "beta")]
    oa = qdelta.recurrent_step(*args, c, d["log_alpha"][0].cuda(), Sa)
    ob = qdelta.recurrent_step(*args, torch.full((N, H), c, device="cuda"), d["log_alpha"][0].cuda(), Sb)
    torch.cuda.synchronize()
    assert torch.equal(oa, ob) and torch.equal(Sa, Sb)
    ref_in = {key: d[key].transpose(0, 1).contiguous() for key in ("q", "k", "v", "beta", "log_alpha")}
    ref_in.update(lam=torch.full((N, 1, H), c), initial_state=S, cu_seqlens=None)
    o_ref, S_ref = oracle_fwd(ref_in)
    assert normwise(f64(oa.cpu()[:, None]), o_ref) <= TOL["bf16"]
    assert normwise(f64(Sa.cpu()), S_ref) <= TOL["bf16"]


@pytest.mark.parametrize("c", [0.2, 1.0])
@pytest.mark.parametrize("varlen", [False, True])
def test_recurrent_fwd_constant_lambda(c, varlen):
    if varlen:
        d = synth.make(1, 0, 2, 128, 128, "bf16", "G2", seed=164, s0=True, lengths=[40, 1, 90])
    else:
        d = synth.make(3, 50, 2, 128, 128, "bf16", "G2", seed=165, s0=True)
    dc = _filled(d, c)
    args = (dev(d["q"]), dev(d["k"]), dev(d["v"]), dev(d["beta"]))
    o, Sf = qdelta.recurrent_fwd(*args, c, dev(d["log_alpha"]), dev(d["initial_state"]),
                                 cu_seqlens=dev(d["cu_seqlens"]))
    o_t, Sf_t = qdelta.recurrent_fwd(*args, dev(dc["lam"]), dev(d["log_alpha"]), dev(d["initial_state"]),
                                     cu_seqlens=dev(d["cu_seqlens"]))
    torch.cuda.synchronize()
    assert torch.equal(o, o_t) and torch.equal(Sf, Sf_t)
    e = fwd_errors(dc, o, Sf)
    assert all(v <= TOL["bf16"] for v in e.values()), e
