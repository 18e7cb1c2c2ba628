"""Pins of the CPU oracle against what the paper and the mathematics fix.

The paper prints no worked numeric example, so every pin here is a closed
form, an exact special case, an invariant, an independent exact evaluation, or
a finite-difference derivative.  Each is chosen so that a plausible slip in the
oracle (a dropped lambda term, a wrong sign, the pre-update state in the
read-out, a transposed operand, a missing decay) fails at least one of them.
"""
from fractions import Fraction as Fr

import numpy as np
import pytest

from oracle import chunk, deltanet, exact, recurrent


def _rand_inputs(rng, B, T, H, dk, dv, decay=True, s0=True, unit=True):
    q = rng.standard_normal((B, T, H, dk))
    k = rng.standard_normal((B, T, H, dk))
    if unit:
        q /= np.linalg.norm(q, axis=-1, keepdims=True)
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, T, H, dv))
    beta = 1 / (1 + np.exp(-rng.standard_normal((B, T, H))))
    lam = 1 / (1 + np.exp(-rng.standard_normal((B, T, H))))
    la = np.log(1 / (1 + np.exp(-rng.normal(2.0, 1.0, (B, T, H))))) if decay else None
    S0 = rng.normal(0, 0.3, (B, H, dv, dk)) if s0 else None
    return q, k, v, beta, lam, la, S0


def _dyadic(rng, shape, den=8, lo=-8, hi=8):
    return rng.integers(lo, hi + 1, size=shape) / den


# ---------------------------------------------------------------- exact pins

def _tiny_rational_case(seed=0, T=6, dk=3, dv=2):
    rng = np.random.default_rng(seed)
    q = _dyadic(rng, (T, dk))
    k = _dyadic(rng, (T, dk))
    v = _dyadic(rng, (T, dv))
    beta = rng.integers(1, 8, size=T) / 8
    lam = rng.integers(0, 9, size=T) / 8
    alpha = rng.integers(1, 9, size=T) / 8
    S0 = _dyadic(rng, (dv, dk), den=4)
    return q, k, v, beta, lam, alpha, S0


def test_exact_dense_product_equals_value_decomposition():
    """Sec. 3.1 value decomposition == explicit transition-matrix product, exactly."""
    for seed in range(4):
        q, k, v, beta, lam, alpha, S0 = _tiny_rational_case(seed)
        conv = lambda a: [[Fr(x) for x in row] for row in a]
        args = (conv(q), conv(k), conv(v), [Fr(x) for x in beta], [Fr(x) for x in lam],
                [Fr(x) for x in alpha], conv(S0))
        o1, S1 = exact.dense_product(*args)
        o2, S2 = exact.closed_form(*args)
        assert o1 == o2
        assert S1 == S2


def test_oracle_matches_exact_rational_brute_force():
    for seed in range(6):
        q, k, v, beta, lam, alpha, S0 = _tiny_rational_case(seed, T=8, dk=4, dv=3)
        conv = lambda a: [[Fr(x) for x in row] for row in a]
        o_ex, S_ex = exact.dense_product(conv(q), conv(k), conv(v), [Fr(x) for x in beta],
                                         [Fr(x) for x in lam], [Fr(x) for x in alpha], conv(S0))
        o_ex = np.array([[float(x) for x in row] for row in o_ex])
        S_ex = np.array([[float(x) for x in row] for row in S_ex])
        o, Sf = recurrent.fwd(q[None, :, None], k[None, :, None], v[None, :, None],
                              beta[None, :, None], lam[None, :, None],
                              alpha=alpha[None, :, None], initial_state=S0[None, None])
        scale = max(1.0, np.abs(o_ex).max())
        assert np.abs(o[0, :, 0] - o_ex).max() <= 1e-14 * scale
        assert np.abs(Sf[0, 0] - S_ex).max() <= 1e-14 * max(1.0, np.abs(S_ex).max())


def test_golden_exact_fixture():
    """Exact rational outputs stored by tests/golden/make_golden.py (oracle.exact only)."""
    import json, os
    path = os.path.join(os.path.dirname(__file__), "golden", "exact_T5_dk3_dv2.json")
    with open(path) as f:
        g = json.load(f)
    inp = g["inputs"]
    F = lambda x: Fr(x)
    conv = lambda a: [[F(x) for x in row] for row in a]
    o, S = exact.dense_product(conv(inp["q"]), conv(inp["k"]), conv(inp["v"]),
                               [F(x) for x in inp["beta"]], [F(x) for x in inp["lam"]],
                               [F(x) for x in inp["alpha"]], conv(inp["S0"]))
    assert [[str(x) for x in row] for row in o] == g["o"]
    assert [[str(x) for x in row] for row in S] == g["S_final"]
    # and the fp64 oracle on the same (dyadic, exactly representable) inputs
    f = lambda a: np.array([[float(Fr(x)) for x in row] for row in a])
    o64, S64 = recurrent.fwd(f(inp["q"])[None, :, None], f(inp["k"])[None, :, None],
                             f(inp["v"])[None, :, None],
                             np.array([float(Fr(x)) for x in inp["beta"]])[None, :, None],
                             np.array([float(Fr(x)) for x in inp["lam"]])[None, :, None],
                             alpha=np.array([float(Fr(x)) for x in inp["alpha"]])[None, :, None],
                             initial_state=f(inp["S0"])[None, None])
    assert np.allclose(o64[0, :, 0], f(g["o"]), rtol=0, atol=1e-13)
    assert np.allclose(S64[0, 0], f(g["S_final"]), rtol=0, atol=1e-13)


def test_hand_worked_scalar_and_matrix_steps():
    """Two steps worked by hand from Eq. (qdelta_decay), d_k = d_v = 1.

    step 1: S0=1/2, q=1, k=1, v=2, beta=1/2, lambda=1/2, alpha=1/2
            x = 3/2;  S1 = 1/2*1/2*(1 - 1/2*3/2*1) + 1/2*2*1 = 1/16 + 1 = 17/16; o1 = 17/16
    step 2: q=-1, k=1/2, v=1, beta=1, lambda=1, alpha=1
            x = -1/2; S2 = 17/16*(1 + 1/4) + 1/2 = 85/64 + 32/64 = 117/64; o2 = -117/64
    """
    q = np.array([1.0, -1.0]); k = np.array([1.0, 0.5]); v = np.array([2.0, 1.0])
    beta = np.array([0.5, 1.0]); lam = np.array([0.5, 1.0]); alpha = np.array([0.5, 1.0])
    o, S = recurrent.fwd(q[None, :, None, None], k[None, :, None, None], v[None, :, None, None],
                         beta[None, :, None], lam[None, :, None], alpha=alpha[None, :, None],
                         initial_state=np.array([[[[0.5]]]]))
    assert o[0, :, 0, 0].tolist() == [17 / 16, -117 / 64]
    assert S[0, 0, 0, 0] == 117 / 64
    # d_k = d_v = 2, one step, identity initial state:
    #   x = k + q = (1,1); S0 x = (1,1); e = v - S0 x = (2,3)
    #   S1 = I + 1/2 (2,3)^T (1,0) = [[2,0],[3/2,1]];  o1 = S1 q = (0, 1)
    o, S = recurrent.fwd(np.array([0.0, 1.0])[None, None, None], np.array([1.0, 0.0])[None, None, None],
                         np.array([3.0, 4.0])[None, None, None], np.array([[[0.5]]]),
                         np.array([[[1.0]]]), initial_state=np.eye(2)[None, None])
    assert S[0, 0].tolist() == [[2.0, 0.0], [1.5, 1.0]]
    assert o[0, 0, 0].tolist() == [0.0, 1.0]


# ---------------------------------------------------------------- reductions

@pytest.mark.parametrize("decay", [False, True])
def test_lambda_zero_reduces_to_deltanet_and_gated_deltanet(decay):
    rng = np.random.default_rng(1)
    q, k, v, beta, lam, la, S0 = _rand_inputs(rng, 1, 40, 2, 8, 6, decay=decay)
    lam = np.zeros_like(lam)
    o, Sf = recurrent.fwd(q, k, v, beta, lam, la, S0)
    for h in range(2):
        a = None if la is None else np.exp(la[0, :, h])
        o_ref, S_ref = deltanet.gated_delta(q[0, :, h], k[0, :, h], v[0, :, h], beta[0, :, h], a, S0[0, h])
        assert np.abs(o[0, :, h] - o_ref).max() < 1e-12
        assert np.abs(Sf[0, h] - S_ref).max() < 1e-12


def test_lambda_nonzero_differs_from_deltanet():
    """Guards against an oracle that silently ignores lambda."""
    rng = np.random.default_rng(2)
    q, k, v, beta, lam, la, S0 = _rand_inputs(rng, 1, 20, 1, 8, 6)
    o, _ = recurrent.fwd(q, k, v, beta, lam, la, S0)
    o_ref, _ = deltanet.gated_delta(q[0, :, 0], k[0, :, 0], v[0, :, 0], beta[0, :, 0],
                                    np.exp(la[0, :, 0]), S0[0, 0])
    assert np.abs(o[0, :, 0] - o_ref).max() > 1e-3


def test_beta_zero_keeps_state_or_only_decays():
    rng = np.random.default_rng(3)
    q, k, v, beta, lam, la, S0 = _rand_inputs(rng, 2, 30, 2, 8, 5)
    beta = np.zeros_like(beta)
    o, Sf = recurrent.fwd(q, k, v, beta, lam, None, S0)
    assert np.array_equal(Sf, S0)
    assert np.allclose(o, np.einsum("bhvk,bthk->bthv", S0, q), atol=1e-15)
    o, Sf = recurrent.fwd(q, k, v, beta, lam, la, S0)
    cum = np.exp(np.cumsum(la, axis=1))                                # prod_{j<=t} alpha_j
    assert np.allclose(Sf, np.exp(la.sum(axis=1))[:, :, None, None] * S0, rtol=1e-13, atol=0)
    assert np.allclose(o, cum[..., None] * np.einsum("bhvk,bthk->bthv", S0, q), rtol=1e-12, atol=1e-15)


def test_alpha_zero_resets_memory():
    """alpha_t = 0 erases the past: S_t = beta_t v_t k_t^T, o_t = beta_t (k_t . q_t) v_t."""
    rng = np.random.default_rng(4)
    q, k, v, beta, lam, _, S0 = _rand_inputs(rng, 1, 5, 1, 6, 4)
    alpha = np.ones((1, 5, 1)); alpha[0, 4, 0] = 0.0
    o, Sf = recurrent.fwd(q, k, v, beta, lam, alpha=alpha, initial_state=S0)
    t = 4
    assert np.allclose(Sf[0, 0], beta[0, t, 0] * np.outer(v[0, t, 0], k[0, t, 0]), atol=1e-15)
    assert np.allclose(o[0, t, 0], beta[0, t, 0] * (k[0, t, 0] @ q[0, t, 0]) * v[0, t, 0], atol=1e-15)


def test_readout_uses_updated_state():
    """One token from a zero state: S_1 = beta v k^T, so o_1 = beta (k.q) v (non-zero);
    a read-out from the previous state would give 0."""
    rng = np.random.default_rng(5)
    q, k, v, beta, lam, la, _ = _rand_inputs(rng, 1, 1, 1, 8, 4)
    o, _ = recurrent.fwd(q, k, v, beta, lam, la)
    assert np.allclose(o[0, 0, 0], beta[0, 0, 0] * (k[0, 0, 0] @ q[0, 0, 0]) * v[0, 0, 0], atol=1e-15)


def test_lemma1_contraction_identity_with_decay():
    """v_t - S_t x_t = (1 - beta_t a_t)(v_t - alpha_t S_{t-1} x_t), a_t = k_t . x_t
    (Lemma 1, extended to the decayed rule), checked at every step."""
    rng = np.random.default_rng(6)
    q, k, v, beta, lam, la, S0 = _rand_inputs(rng, 1, 25, 1, 8, 5)
    S = S0[0, 0]
    worst = 0.0
    for t in range(25):
        sl = slice(t, t + 1)
        _, Sn = recurrent.fwd(q[:, sl], k[:, sl], v[:, sl], beta[:, sl], lam[:, sl], la[:, sl],
                              S[None, None])
        Sn = Sn[0, 0]
        x = k[0, t, 0] + lam[0, t, 0] * q[0, t, 0]
        a = k[0, t, 0] @ x
        lhs = v[0, t, 0] - Sn @ x
        rhs = (1 - beta[0, t, 0] * a) * (v[0, t, 0] - np.exp(la[0, t, 0]) * (S @ x))
        worst = max(worst, np.abs(lhs - rhs).max())
        # L2-normalised q, k and beta, lambda in (0,1) keep beta*a in (0, 2)
        assert 0 < beta[0, t, 0] * a < 2
        S = Sn
    assert worst < 1e-13


def test_linearity_in_values_and_initial_state():
    rng = np.random.default_rng(7)
    q, k, v1, beta, lam, la, S1 = _rand_inputs(rng, 2, 33, 2, 8, 6)
    v2 = rng.standard_normal(v1.shape)
    S2 = rng.standard_normal(S1.shape)
    a, b = 0.7, -1.3
    o1, F1 = recurrent.fwd(q, k, v1, beta, lam, la, S1)
    o2, F2 = recurrent.fwd(q, k, v2, beta, lam, la, S2)
    o3, F3 = recurrent.fwd(q, k, a * v1 + b * v2, beta, lam, la, a * S1 + b * S2)
    assert np.abs(o3 - (a * o1 + b * o2)).max() < 1e-12
    assert np.abs(F3 - (a * F1 + b * F2)).max() < 1e-12


def test_continuation_and_varlen_equal_separate_runs():
    rng = np.random.default_rng(8)
    q, k, v, beta, lam, la, S0 = _rand_inputs(rng, 1, 50, 2, 8, 6)
    o, Sf = recurrent.fwd(q, k, v, beta, lam, la, S0)
    a = slice(0, 21); b = slice(21, 50)
    oa, Sa = recurrent.fwd(q[:, a], k[:, a], v[:, a], beta[:, a], lam[:, a], la[:, a], S0)
    ob, Sb = recurrent.fwd(q[:, b], k[:, b], v[:, b], beta[:, b], lam[:, b], la[:, b], Sa)
    assert np.array_equal(np.concatenate([oa, ob], axis=1), o)
    assert np.array_equal(Sb, Sf)
    # packed: two sequences [0,21) and [21,50), each from its own initial state
    S0b = rng.standard_normal(S0.shape)
    S0s = np.concatenate([S0, S0b])
    op, Sp = recurrent.fwd(q[0], k[0], v[0], beta[0], lam[0], la[0], S0s, cu_seqlens=[0, 21, 50])
    ob2, Sb2 = recurrent.fwd(q[:, b], k[:, b], v[:, b], beta[:, b], lam[:, b], la[:, b], S0b)
    assert np.array_equal(op[:21], oa[0]) and np.array_equal(op[21:], ob2[0])
    assert np.array_equal(Sp[0], Sa[0]) and np.array_equal(Sp[1], Sb2[0])


def test_empty_sequences_in_packed_batch():
    rng = np.random.default_rng(9)
    q, k, v, beta, lam, la, _ = _rand_inputs(rng, 1, 10, 1, 4, 3, s0=False)
    S0 = rng.standard_normal((3, 1, 3, 4))
    o, Sf = recurrent.fwd(q[0], k[0], v[0], beta[0], lam[0], la[0], S0, cu_seqlens=[0, 0, 10, 10])
    assert np.array_equal(Sf[0], S0[0]) and np.array_equal(Sf[2], S0[2])


# ---------------------------------------------------------------- chunk algebra

def test_chunk_form_equals_recurrence_for_every_chunk_size():
    rng = np.random.default_rng(10)
    T = 37
    q, k, v, beta, lam, la, S0 = _rand_inputs(rng, 1, T, 1, 6, 5)
    o, Sf = recurrent.fwd(q, k, v, beta, lam, la, S0)
    for C in range(1, T + 1):
        oc, Sc = chunk.fwd(q, k, v, beta, lam, la, S0, C=C)
        assert np.abs(oc - o).max() < 1e-12 * max(1, np.abs(o).max()), C
        assert np.abs(Sc - Sf).max() < 1e-12 * max(1, np.abs(Sf).max()), C


@pytest.mark.parametrize("decay", [False, True])
def test_chunk_form_equals_recurrence_tiny_layer_shape(decay):
    """The fp32 tiny-layer shape (T=256, H=2, d=64) for several chunk sizes,
    including ones that do not divide T."""
    rng = np.random.default_rng(11)
    q, k, v, beta, lam, la, S0 = _rand_inputs(rng, 1, 256, 2, 64, 64, decay=decay)
    o, Sf = recurrent.fwd(q, k, v, beta, lam, la, S0)
    for C in (1, 7, 16, 48, 64, 100, 256):
        oc, Sc = chunk.fwd(q, k, v, beta, lam, la, S0, C=C)
        assert np.abs(oc - o).max() <= 1e-12 * np.abs(o).max(), C
        assert np.abs(Sc - Sf).max() <= 1e-12 * np.abs(Sf).max(), C


def test_single_solve_W_equals_papers_two_solve_form():
    """W = (I+A)^{-1} diag(beta) diag(g) X  ==  diag(g) W_paper of Eq. (qdelta_chunk_U)."""
    rng = np.random.default_rng(12)
    q, k, v, beta, lam, la, _ = _rand_inputs(rng, 1, 16, 1, 6, 5)
    st = chunk._chunk_setup(q[0, :, 0], k[0, :, 0], v[0, :, 0], beta[0, :, 0], lam[0, :, 0], la[0, :, 0])
    Wp = chunk.paper_two_solve_W(k[0, :, 0], q[0, :, 0], beta[0, :, 0], lam[0, :, 0], la[0, :, 0])
    assert np.abs(st["W"] - Wp).max() < 1e-13


def test_chunk_transfer_is_affine():
    """S' = S (g_C I - W^T Kbar) + U^T Kbar for every entry state S."""
    rng = np.random.default_rng(13)
    q, k, v, beta, lam, la, _ = _rand_inputs(rng, 1, 16, 1, 6, 5)
    Q, K, V = q[0, :, 0], k[0, :, 0], v[0, :, 0]
    st = chunk._chunk_setup(Q, K, V, beta[0, :, 0], lam[0, :, 0], la[0, :, 0])
    Kbar = np.exp(st["b"][-1] - st["b"])[:, None] * K
    for _ in range(3):
        S = rng.standard_normal((5, 6))
        _, S1, _ = chunk.fwd_unit(Q, K, V, beta[0, :, 0], lam[0, :, 0], la[0, :, 0], S, 16)
        S2 = S @ (st["g"][-1] * np.eye(6) - st["W"].T @ Kbar) + st["U"].T @ Kbar
        assert np.abs(S1 - S2).max() < 1e-13


# ---------------------------------------------------------------- gradients

def _loss(q, k, v, beta, lam, alpha, S0, dO, dSf):
    o, Sf = recurrent.fwd(q, k, v, beta, lam, alpha=alpha, initial_state=S0)
    return float(np.sum(o * dO) + np.sum(Sf * dSf))


def test_bptt_matches_central_finite_differences():
    rng = np.random.default_rng(14)
    q, k, v, beta, lam, la, S0 = _rand_inputs(rng, 1, 11, 1, 5, 4)
    alpha = np.exp(la)
    dO = rng.standard_normal(v.shape)
    dSf = rng.standard_normal(S0.shape)
    g = recurrent.bwd(q, k, v, beta, lam, alpha=alpha, initial_state=S0, d_o=dO, d_final_state=dSf)
    args = dict(q=q, k=k, v=v, beta=beta, lam=lam, alpha=alpha, S0=S0)
    names = dict(q="dq", k="dk", v="dv", beta="dbeta", lam="dlam", alpha="dalpha", S0="d_initial_state")
    h = 1e-6
    for name, gname in names.items():
        x = args[name]
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp = x.copy(); xp[idx] += h
            xm = x.copy(); xm[idx] -= h
            a1 = dict(args); a1[name] = xp
            a2 = dict(args); a2[name] = xm
            fd[idx] = (_loss(dO=dO, dSf=dSf, **a1) - _loss(dO=dO, dSf=dSf, **a2)) / (2 * h)
        err = np.abs(fd - g[gname]).max() / max(1e-3, np.abs(fd).max())
        assert err < 1e-7, (name, err)


def test_log_alpha_gradient_is_alpha_times_alpha_gradient():
    rng = np.random.default_rng(15)
    q, k, v, beta, lam, la, S0 = _rand_inputs(rng, 1, 9, 1, 4, 3)
    dO = rng.standard_normal(v.shape)
    g = recurrent.bwd(q, k, v, beta, lam, la, S0, d_o=dO)
    h = 1e-6
    fd = np.zeros_like(la)
    for idx in np.ndindex(la.shape):
        lp = la.copy(); lp[idx] += h
        lm = la.copy(); lm[idx] -= h
        fp = np.sum(recurrent.fwd(q, k, v, beta, lam, lp, S0)[0] * dO)
        fm = np.sum(recurrent.fwd(q, k, v, beta, lam, lm, S0)[0] * dO)
        fd[idx] = (fp - fm) / (2 * h)
    assert np.abs(fd - g["dlog_alpha"]).max() < 1e-7 * max(1, np.abs(fd).max())


@pytest.mark.parametrize("C,T,decay", [(6, 23, True), (64, 150, True), (64, 130, False), (1, 9, True)])
def test_chunk_backward_equals_bptt(C, T, decay):
    rng = np.random.default_rng(16)
    q, k, v, beta, lam, la, S0 = _rand_inputs(rng, 1, T, 2, 8, 6, decay=decay)
    dO = rng.standard_normal(v.shape)
    dSf = rng.standard_normal(S0.shape)
    g = recurrent.bwd(q, k, v, beta, lam, la, S0, d_o=dO, d_final_state=dSf)
    gc = chunk.bwd(q, k, v, beta, lam, la, S0, d_o=dO, d_final_state=dSf, C=C)
    for key in ("dq", "dk", "dv", "dbeta", "dlam", "d_initial_state") + (("dlog_alpha",) if decay else ()):
        ref = g[key]
        assert np.abs(gc[key] - ref).max() <= 1e-11 * max(1, np.abs(ref).max()), key


def test_varlen_backward_equals_separate():
    rng = np.random.default_rng(17)
    q, k, v, beta, lam, la, _ = _rand_inputs(rng, 1, 40, 2, 6, 5, s0=False)
    S0 = rng.standard_normal((2, 2, 5, 6))
    dO = rng.standard_normal(v.shape)
    cu = [0, 17, 40]
    g = recurrent.bwd(q[0], k[0], v[0], beta[0], lam[0], la[0], S0, d_o=dO[0], cu_seqlens=cu)
    for n in range(2):
        sl = slice(cu[n], cu[n + 1])
        gs = recurrent.bwd(q[:, sl], k[:, sl], v[:, sl], beta[:, sl], lam[:, sl], la[:, sl],
                           S0[n:n + 1], d_o=dO[:, sl])
        assert np.array_equal(g["dq"][sl], gs["dq"][0])
        assert np.array_equal(g["dlog_alpha"][sl], gs["dlog_alpha"][0])
        assert np.array_equal(g["d_initial_state"][n], gs["d_initial_state"][0])
