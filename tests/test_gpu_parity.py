"""GPU parity of the HIP path against the fp64 oracle at sizes that span
several chunks and a ragged tail, in every gate mode, plus invariants.

Tolerances: normwise max error max|got-ref|/max|ref| per output tensor,
1e-4 for fp32 inputs and 2e-2 for bf16 inputs (fp32 accumulation)."""
import numpy as np
import pytest
import torch

from paper_2606_08804_amd import qdelta, synth
from tests.gpu_helpers import (TOL, bwd_errors, dev, f64, fwd_errors, gpu_bwd, gpu_fwd, normwise,
                               oracle_fwd)

pytestmark = pytest.mark.gpu

GATES = ["G1", "G2", "G3"]


def _check(errs, tol, what):
    bad = {k: v for k, v in errs.items() if not (v <= tol)}
    assert not bad, f"{what}: {errs}"


@pytest.mark.parametrize("gate", GATES)
@pytest.mark.parametrize("Dv", [64, 128, 256])
def test_fwd_fp32(gate, Dv):
    d = synth.make(2, 200, 2, 64, Dv, "f32", gate, seed=101, s0=True)
    o, Sf, _ = gpu_fwd(d)
    _check(fwd_errors(d, o, Sf), TOL["f32"], f"fwd fp32 {gate} Dv={Dv}")


@pytest.mark.parametrize("gate", GATES)
@pytest.mark.parametrize("Dk,Dv", [(128, 128), (128, 256), (64, 64), (128, 64), (64, 256), (64, 128)])
def test_fwd_bf16(gate, Dk, Dv):
    d = synth.make(2, 300, 2, Dk, Dv, "bf16", gate, seed=102, s0=True)
    o, Sf, _ = gpu_fwd(d)
    _check(fwd_errors(d, o, Sf), TOL["bf16"], f"fwd bf16 {gate} Dk={Dk} Dv={Dv}")


def test_tiny_fp32_layer_workload():
    """The tiny fp32 layer: B=1, T=256, H=2, d=64, zero initial state."""
    for gate in ("G1", "G2"):
        d = synth.make_workload(1, gate)
        o, Sf, _ = gpu_fwd(d)
        _check(fwd_errors(d, o, Sf), TOL["f32"], f"tiny fp32 {gate}")


@pytest.mark.parametrize("T", [1, 63, 64, 65, 127, 129])
def test_fwd_edge_lengths(T):
    for dt in ("f32", "bf16"):
        d = synth.make(1, T, 1, 64, 64, dt, "G2", seed=103 + T, s0=True)
        o, Sf, _ = gpu_fwd(d)
        _check(fwd_errors(d, o, Sf), TOL[dt], f"fwd {dt} T={T}")


def test_fwd_empty_sequence_passes_state_through():
    d = synth.make(2, 0, 2, 64, 64, "bf16", "G2", seed=104, s0=True)
    o, Sf, _ = gpu_fwd(d)
    assert o.shape == (2, 0, 2, 64)
    assert torch.equal(Sf.cpu(), d["initial_state"])


@pytest.mark.parametrize("Dk,Dv,B,H,T", [(128, 256, 4, 32, 130), (128, 128, 8, 32, 100), (64, 64, 16, 32, 70)])
def test_wide_value_tiles(Dk, Dv, B, H, T):
    """Enough (sequence, head) units that the scans take 64-row value tiles
    (units x Dv/64 >= 2 x 256 CUs), forward and backward, ragged last chunk."""
    d = synth.make(B, T, H, Dk, Dv, "bf16", "G3", seed=110 + Dv, s0=True, with_do=True)
    o, Sf, saved = gpu_fwd(d, save_states=True)
    _check(fwd_errors(d, o, Sf), TOL["bf16"], f"fwd wide tiles Dk={Dk} Dv={Dv}")
    g = gpu_bwd(d, saved)
    _check(bwd_errors(d, g), TOL["bf16"], f"bwd wide tiles Dk={Dk} Dv={Dv}")


@pytest.mark.parametrize("dt,B,H,T", [("bf16", 3, 5, 950), ("f32", 1, 3, 700), ("bf16", 1, 7, 64 * 8 * 3)])
def test_odd_head_counts_and_slot_tails(dt, B, H, T):
    """Head counts that are not powers of two and slot counts that are not
    multiples of 8 (the preparation and intra kernels hand the heads of each
    group of eight slots to one XCD and walk the remaining slots in plain
    order; 24 slots with 7 heads leave no tail), forward and backward."""
    d = synth.make(B, T, H, 64, 64, dt, "G2", seed=140 + H, s0=True, with_do=True)
    o, Sf, saved = gpu_fwd(d, save_states=True)
    _check(fwd_errors(d, o, Sf), TOL[dt], f"fwd {dt} H={H} T={T}")
    g = gpu_bwd(d, saved)
    _check(bwd_errors(d, g), TOL[dt], f"bwd {dt} H={H} T={T}")


@pytest.mark.parametrize("gate", GATES)
@pytest.mark.parametrize("Dv", [64, 128, 256])
def test_bwd_fp32(gate, Dv):
    d = synth.make(2, 150, 2, 64, Dv, "f32", gate, seed=105, s0=True, with_do=True)
    _, _, saved = gpu_fwd(d, save_states=True)
    dSf = torch.from_numpy(np.random.default_rng(5).standard_normal((2, 2, Dv, 64)).astype(np.float32))
    g = gpu_bwd(d, saved, d_final_state=dSf)
    _check(bwd_errors(d, g, dSf), TOL["f32"], f"bwd fp32 {gate} Dv={Dv}")


# every (Dk, Dv) instantiation of the bf16 kernels
BF16_DIMS = [(128, 128), (128, 256), (64, 64), (128, 64), (64, 256), (64, 128)]


@pytest.mark.parametrize("gate", GATES)
@pytest.mark.parametrize("Dk,Dv", BF16_DIMS)
def test_bwd_bf16(gate, Dk, Dv):
    d = synth.make(2, 200, 2, Dk, Dv, "bf16", gate, seed=106, s0=True, with_do=True)
    _, _, saved = gpu_fwd(d, save_states=True)
    g = gpu_bwd(d, saved)
    _check(bwd_errors(d, g), TOL["bf16"], f"bwd bf16 {gate} Dk={Dk} Dv={Dv}")


@pytest.mark.parametrize("gate", ["G1", "G3"])
@pytest.mark.parametrize("Dk,Dv", [(128, 128), (64, 256)])
def test_bwd_bf16_final_state_gradient(gate, Dk, Dv):
    """A non-zero gradient of the final state enters the backward scan's
    accumulator at the last chunk (bf16 activations, fp32 state gradient)."""
    d = synth.make(2, 170, 2, Dk, Dv, "bf16", gate, seed=122, s0=True, with_do=True)
    _, _, saved = gpu_fwd(d, save_states=True)
    dSf = torch.from_numpy(np.random.default_rng(13).standard_normal((2, 2, Dv, Dk)).astype(np.float32))
    g = gpu_bwd(d, saved, d_final_state=dSf)
    _check(bwd_errors(d, g, dSf), TOL["bf16"], f"bwd bf16 dS_final {gate} Dk={Dk} Dv={Dv}")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("gate", ["G1", "G2", "G3"])
def test_beta_zero_closed_form(dt, gate):
    """beta = 0 writes nothing: the state only decays, S_t = (prod_{j<=t} alpha_j) S_0
    (S_t = S_0 without decay) and o_t = S_t q_t.  Checked against that closed
    form (fp64, independent of the oracle) and the oracle, forward and backward."""
    D = 64 if dt == "f32" else 128
    # with G2's decay (mean log alpha -0.81) the state leaves the fp32 range
    # after about 100 tokens, so that mode runs a shorter sequence
    T = 40 if gate == "G2" else 150
    d = synth.make(2, T, 2, D, D, dt, gate, seed=123, s0=True, with_do=True)
    d = dict(d, beta=torch.zeros_like(d["beta"]))
    o, Sf, saved = gpu_fwd(d, save_states=True)
    S0 = f64(d["initial_state"])                                   # [N, H, Dv, Dk]
    cum = (np.zeros(d["beta"].shape) if d["log_alpha"] is None
           else np.cumsum(f64(d["log_alpha"]), axis=1))            # [B, T, H]
    decay = np.exp(cum)
    S_T = decay[:, -1, :, None, None] * S0
    o_ref = decay[..., None] * np.einsum("nhvk,nthk->nthv", S0, f64(d["q"]))
    tol = TOL[dt]
    assert normwise(f64(Sf.cpu()), S_T) <= tol
    assert normwise(f64(o.cpu()), o_ref) <= tol
    _check(fwd_errors(d, o, Sf), tol, f"beta=0 fwd {dt} {gate}")
    g = gpu_bwd(d, saved)
    _check(bwd_errors(d, g), tol, f"beta=0 bwd {dt} {gate}")


@pytest.mark.parametrize("gate", ["G1", "G3"])
def test_bwd_matches_finite_differences_of_gpu_forward(gate):
    """End-to-end gradient check that does not go through the oracle: the
    directional derivative of L = <dO, o> + <dS_T, S_T>, computed by central
    differences of the GPU forward (fp32), equals <grad, u> from the GPU
    backward for a random direction u in each input."""
    d = synth.make(1, 70, 1, 64, 64, "f32", gate, seed=121, s0=True, with_do=True)
    dSf = torch.from_numpy(np.random.default_rng(11).standard_normal((1, 1, 64, 64)).astype(np.float32))
    _, _, saved = gpu_fwd(d, save_states=True)
    g = gpu_bwd(d, saved, d_final_state=dSf)
    dO64, dSf64 = f64(d["d_o"]), f64(dSf)

    def loss(dd):
        o, Sf, _ = gpu_fwd(dd)
        return float((f64(o.cpu()) * dO64).sum() + (f64(Sf.cpu()) * dSf64).sum())

    rng = np.random.default_rng(12)
    names = {"q": "dq", "k": "dk", "v": "dv", "beta": "dbeta", "lam": "dlam", "initial_state": "d_initial_state"}
    if d["log_alpha"] is not None:
        names["log_alpha"] = "dlog_alpha"
    h = 1e-2
    for key, gkey in names.items():
        # a perturbation of about 1% of the input's own scale
        scale = float(d[key].pow(2).mean().sqrt()) + 1e-3
        u = torch.from_numpy((scale * rng.standard_normal(tuple(d[key].shape))).astype(np.float32))
        plus, minus = dict(d), dict(d)
        plus[key] = d[key] + h * u
        minus[key] = d[key] - h * u
        fd = (loss(plus) - loss(minus)) / (2 * h)
        an = float((f64(g[gkey].cpu()) * f64(u)).sum())
        assert abs(fd - an) <= 1e-2 * max(abs(an), 1e-3), (key, fd, an)


def test_bwd_without_saved_states_matches_with():
    d = synth.make(1, 190, 2, 128, 128, "bf16", "G2", seed=107, s0=True, with_do=True)
    _, _, saved = gpu_fwd(d, save_states=True)
    g1 = gpu_bwd(d, saved)
    g2 = gpu_bwd(d, None)
    for key in g1:
        if g1[key] is not None:
            assert torch.equal(g1[key], g2[key]), key


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_varlen_fwd_bwd(dt):
    lengths = [5, 64, 130, 0, 71, 1, 128]
    Dk = 64
    Dv = 128
    d = synth.make(1, 0, 2, Dk, Dv, dt, "G2", seed=108, s0=True, with_do=True, lengths=lengths)
    o, Sf, saved = gpu_fwd(d, save_states=True)
    _check(fwd_errors(d, o, Sf), TOL[dt], f"varlen fwd {dt}")
    g = gpu_bwd(d, saved)
    _check(bwd_errors(d, g), TOL[dt], f"varlen bwd {dt}")


def test_varlen_equals_separate_runs():
    lengths = [70, 3, 200]
    d = synth.make(1, 0, 2, 128, 128, "bf16", "G2", seed=109, s0=True, lengths=lengths)
    o, Sf, _ = gpu_fwd(d)
    cu = d["cu_seqlens"].tolist()
    for n in range(len(lengths)):
        sl = slice(cu[n], cu[n + 1])
        dn = dict(q=d["q"][:, sl].contiguous(), k=d["k"][:, sl].contiguous(), v=d["v"][:, sl].contiguous(),
                  beta=d["beta"][:, sl].contiguous(), lam=d["lam"][:, sl].contiguous(),
                  log_alpha=d["log_alpha"][:, sl].contiguous(),
                  initial_state=d["initial_state"][n:n + 1].contiguous(), cu_seqlens=None)
        on, Sn, _ = gpu_fwd(dn)
        assert torch.equal(on[0].cpu(), o[0, sl].cpu())
        assert torch.equal(Sn[0].cpu(), Sf[n].cpu())


def test_continuation_equals_one_pass():
    d = synth.make(1, 256, 2, 128, 128, "bf16", "G1", seed=110, s0=True)
    o, Sf, _ = gpu_fwd(d)
    a = {k: (v[:, :128].contiguous() if k in ("q", "k", "v", "beta", "lam") else v) for k, v in d.items()}
    b = {k: (v[:, 128:].contiguous() if k in ("q", "k", "v", "beta", "lam") else v) for k, v in d.items()}
    oa, Sa, _ = gpu_fwd(a)
    b["initial_state"] = Sa.cpu()
    ob, Sb, _ = gpu_fwd(b)
    # chunk boundaries coincide, so the two passes do the same arithmetic
    assert torch.equal(torch.cat([oa, ob], dim=1).cpu(), o.cpu())
    assert torch.equal(Sb.cpu(), Sf.cpu())


def test_linearity_in_values_and_initial_state():
    d1 = synth.make(1, 150, 2, 64, 64, "f32", "G2", seed=111, s0=True)
    d2 = synth.make(1, 150, 2, 64, 64, "f32", "G2", seed=112, s0=True)
    d3 = dict(d1)
    d3["v"] = 0.5 * d1["v"] - 2.0 * d2["v"]
    d3["initial_state"] = 0.5 * d1["initial_state"] - 2.0 * d2["initial_state"]
    d2 = dict(d1, v=d2["v"], initial_state=d2["initial_state"])
    o1, S1, _ = gpu_fwd(d1)
    o2, S2, _ = gpu_fwd(d2)
    o3, S3, _ = gpu_fwd(d3)
    assert normwise(f64(o3.cpu()), 0.5 * f64(o1.cpu()) - 2.0 * f64(o2.cpu())) < 1e-5
    assert normwise(f64(S3.cpu()), 0.5 * f64(S1.cpu()) - 2.0 * f64(S2.cpu())) < 1e-5


def test_determinism():
    d = synth.make(2, 200, 2, 128, 128, "bf16", "G2", seed=113, s0=True, with_do=True)
    o1, S1, sv1 = gpu_fwd(d, save_states=True)
    o2, S2, sv2 = gpu_fwd(d, save_states=True)
    assert torch.equal(o1, o2) and torch.equal(S1, S2) and torch.equal(sv1, sv2)
    g1 = gpu_bwd(d, sv1)
    g2 = gpu_bwd(d, sv1)
    for key in g1:
        if g1[key] is not None:
            assert torch.equal(g1[key], g2[key]), key


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("varlen", [False, True])
def test_lambda_none_is_gated_delta_rule(dt, varlen):
    """lam = NULL means lambda == 0: x_t = k_t, the gated delta rule.  The
    result equals the oracle run with lambda = 0 and, bit for bit, the GPU
    path run with an explicit all-zero lambda; no dlam is written."""
    D = 128 if dt == "bf16" else 64
    if varlen:
        d = synth.make(1, 0, 2, D, D, dt, "G3", seed=131, s0=True, with_do=True,
                       lengths=[70, 1, 130, 64])
    else:
        d = synth.make(2, 150, 2, D, D, dt, "G3", seed=131, s0=True, with_do=True)
    d0 = dict(d, lam=torch.zeros_like(d["lam"]))
    dn = dict(d, lam=None)
    o, Sf, saved = gpu_fwd(dn, save_states=True)
    _check(fwd_errors(d0, o, Sf), TOL[dt], f"fwd lam=None {dt}")
    g = gpu_bwd(dn, saved)
    assert g["dlam"] is None
    _check(bwd_errors(d0, g, skip=("dlam",)), TOL[dt], f"bwd lam=None {dt}")
    o0, Sf0, saved0 = gpu_fwd(d0, save_states=True)
    g0 = gpu_bwd(d0, saved0)
    assert torch.equal(o, o0) and torch.equal(Sf, Sf0)
    for key in ("dq", "dk", "dv", "dbeta", "dlog_alpha", "d_initial_state"):
        assert torch.equal(g[key], g0[key]), key


def test_recurrent_step_lambda_none():
    N, H, D = 8, 4, 128
    d = synth.make(1, N, H, D, D, "bf16", "G2", seed=132)
    S = torch.from_numpy(np.random.default_rng(6).normal(0, 0.02, (N, H, D, D)).astype(np.float32))
    Sa, Sb = S.cuda(), S.cuda()
    args = [d[key][0].cuda() for key in ("q", "k", "v", "beta")]
    oa = qdelta.recurrent_step(*args, None, d["log_alpha"][0].cuda(), Sa)
    ob = qdelta.recurrent_step(*args, torch.zeros(N, H, device="cuda"), d["log_alpha"][0].cuda(), Sb)
    torch.cuda.synchronize()
    assert torch.equal(oa, ob) and torch.equal(Sa, Sb)
    ref_in = {key: d[key].transpose(0, 1).contiguous() for key in ("q", "k", "v", "beta", "log_alpha")}
    ref_in.update(lam=torch.zeros(N, 1, H), initial_state=S, cu_seqlens=None)
    o_ref, S_ref = oracle_fwd(ref_in)
    assert normwise(f64(oa.cpu()[:, None]), o_ref) <= TOL["bf16"]
    assert normwise(f64(Sa.cpu()), S_ref) <= TOL["bf16"]


@pytest.mark.parametrize("dt,D", [("bf16", 128), ("f32", 64), ("bf16", 64)])
def test_recurrent_step_parity(dt, D):
    N, H, steps = 8, 4, 5
    d = synth.make(steps, N, H, D, D, dt, "G2", seed=114)
    S = torch.from_numpy(np.random.default_rng(3).normal(0, 0.02, (N, H, D, D)).astype(np.float32))
    Sg = S.cuda()
    outs = []
    for s in range(steps):
        o = qdelta.recurrent_step(d["q"][s].cuda(), d["k"][s].cuda(), d["v"][s].cuda(),
                                  d["beta"][s].cuda(), d["lam"][s].cuda(), d["log_alpha"][s].cuda(), Sg)
        outs.append(o.cpu())
    torch.cuda.synchronize()
    # oracle: the same tokens as N sequences of `steps` tokens
    ref_in = {k: (d[k].transpose(0, 1).contiguous() if d[k] is not None and k not in ("initial_state",) else d[k])
              for k in ("q", "k", "v", "beta", "lam", "log_alpha")}
    ref_in.update(initial_state=S, cu_seqlens=None, d_o=None)
    o_ref, S_ref = oracle_fwd(ref_in)
    o_got = f64(torch.stack(outs, 0).transpose(0, 1))
    tol = TOL[dt]
    assert normwise(o_got, o_ref) <= tol
    assert normwise(f64(Sg.cpu()), S_ref) <= tol


def test_decode_equals_chunk_forward():
    """Successive single-token updates equal one chunk forward over the same tokens."""
    N, H, D, steps = 4, 2, 128, 200
    d = synth.make(steps, N, H, D, D, "bf16", "G1", seed=115)
    S0 = torch.from_numpy(np.random.default_rng(4).normal(0, 0.02, (N, H, D, D)).astype(np.float32))
    Sg = S0.cuda()
    outs = []
    for s in range(steps):
        outs.append(qdelta.recurrent_step(d["q"][s].cuda(), d["k"][s].cuda(), d["v"][s].cuda(),
                                          d["beta"][s].cuda(), d["lam"][s].cuda(), None, Sg))
    seq = {k: d[k].transpose(0, 1).contiguous() for k in ("q", "k", "v", "beta", "lam")}
    seq.update(log_alpha=None, initial_state=S0, cu_seqlens=None)
    o, Sf, _ = gpu_fwd(seq)
    o_dec = torch.stack(outs, 0).transpose(0, 1)
    assert normwise(f64(o_dec.cpu()), f64(o.cpu())) <= TOL["bf16"]
    assert normwise(f64(Sg.cpu()), f64(Sf.cpu())) <= TOL["bf16"]
