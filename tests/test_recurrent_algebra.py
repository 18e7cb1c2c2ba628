"""The regrouping the fully recurrent forward kernel computes, written out in
fp64 and checked against the oracle's recurrence (Sec. 3.3, Eq. qdelta_decay):

* both row dot products use the state before the update:
  o_t = alpha_t S_{t-1} q_t + e_t (k_t . q_t), e_t = beta_t (v_t - alpha_t S_{t-1} x_t);
* the state is held as a scale times stored rows: the decay multiplies the
  scale, the update adds (e_t / scale) k_t^T, the scale is folded back every
  16 tokens, and a token with alpha < 2^-6 takes the explicit update.

A slip in any of these (the updated state in a dot product, the scale applied
twice or not at all, a missed fold) changes o or the final state."""
import numpy as np

from oracle import recurrent

TB = 16


def regrouped(q, k, v, beta, lam, alpha, S0):
    S = S0.copy()
    sc = 1.0
    out = np.zeros((len(q), S.shape[0]))
    for t in range(len(q)):
        pk, pq, kq = S @ k[t], S @ q[t], k[t] @ q[t]
        sq = sc * pq
        e = beta[t] * (v[t] - alpha[t] * (sc * pk + lam[t] * sq))
        out[t] = alpha[t] * sq + e * kq
        if alpha[t] >= 2.0 ** -6:
            sc *= alpha[t]
            S += np.outer(e / sc, k[t])
        else:
            S = sc * alpha[t] * S + np.outer(e, k[t])
            sc = 1.0
        if t % TB == TB - 1 or t == len(q) - 1:
            S *= sc
            sc = 1.0
    return out, S


def test_regrouped_recurrence_equals_oracle():
    rng = np.random.default_rng(7)
    T, dk, dv = 70, 8, 5
    q = rng.standard_normal((T, dk))
    k = rng.standard_normal((T, dk))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    k /= np.linalg.norm(k, axis=1, keepdims=True)
    v = rng.standard_normal((T, dv))
    beta = 1 / (1 + np.exp(-rng.standard_normal(T)))
    lam = 1 / (1 + np.exp(-rng.standard_normal(T)))
    alpha = 1 / (1 + np.exp(-rng.standard_normal(T)))
    alpha[[5, 33, 34]] = [1e-3, 2.0 ** -7, 0.0]       # the explicit-update branch, alpha == 0 included
    S0 = rng.normal(0, 0.3, (dv, dk))
    o, S = regrouped(q, k, v, beta, lam, alpha, S0)
    o_ref, S_ref = recurrent.fwd(q[None, :, None], k[None, :, None], v[None, :, None],
                                 beta[None, :, None], lam[None, :, None], None, S0[None, None],
                                 alpha=alpha[None, :, None])
    assert np.abs(o - o_ref[0, :, 0]).max() <= 1e-12 * np.abs(o_ref).max()
    assert np.abs(S - S_ref[0, 0]).max() <= 1e-12 * np.abs(S_ref).max()


def three_sweep_backward(q, k, v, beta, lam, alpha, S0, dO, dSf):
    """The fully recurrent backward kernel's regrouping, for one (sequence,
    head): a forward sweep storing p_t = S_{t-1} x_t and z_t = dO_t * o_t per
    row; a reverse sweep carrying only the state adjoint G (dv, dbeta,
    dlog alpha, and sum_i e_i G_i), where <G_t, S_{t-1}> comes from the
    per-row scalar F_t = <G_t, S_t> (F_{t-1} = F_t - e s + dp p + z_{t-1},
    alpha <G_t, S_{t-1}> = F_t - e s); a second forward sweep for the column
    sums S_{t-1}^T dO_t and S_{t-1}^T dp_t (dq, dk, dlambda)."""
    T, dk = q.shape
    dv = v.shape[1]
    S = S0.copy()
    P = np.zeros((T, dv))
    Z = np.zeros((T, dv))
    for t in range(T):                                  # sweep A
        x = k[t] + lam[t] * q[t]
        P[t] = S @ x
        e = beta[t] * (v[t] - alpha[t] * P[t])
        S = alpha[t] * S + np.outer(e, k[t])
        Z[t] = dO[t] * (S @ q[t])
    F = (dSf * S).sum(1) + Z[T - 1]
    G = dSf.copy()
    dv_, dbeta, dla = np.zeros((T, dv)), np.zeros(T), np.zeros(T)
    DP, WK = np.zeros((T, dv)), np.zeros((T, dk))
    for t in range(T - 1, -1, -1):                      # sweep B
        x = k[t] + lam[t] * q[t]
        G = G + np.outer(dO[t], q[t])
        s = G @ k[t]
        u = v[t] - alpha[t] * P[t]
        e = beta[t] * u
        dp = -alpha[t] * beta[t] * s
        dv_[t] = beta[t] * s
        DP[t] = dp
        dbeta[t] = (u * s).sum()
        dla[t] = (F - e * s + dp * P[t]).sum()
        F = F - e * s + dp * P[t] + (Z[t - 1] if t > 0 else 0.0)
        WK[t] = e @ G
        G = alpha[t] * G + np.outer(dp, x)
    dS0 = G
    S = S0.copy()
    dq, dk_, dlam = np.zeros((T, dk)), np.zeros((T, dk)), np.zeros(T)
    for t in range(T):                                  # sweep C
        x = k[t] + lam[t] * q[t]
        p = S @ x
        e = beta[t] * (v[t] - alpha[t] * p)
        w1, w2, c = S.T @ dO[t], S.T @ DP[t], dO[t] @ e
        dq[t] = alpha[t] * w1 + c * k[t] + lam[t] * w2
        dk_[t] = WK[t] + w2
        dlam[t] = q[t] @ w2
        S = alpha[t] * S + np.outer(e, k[t])
    return dict(dq=dq, dk=dk_, dv=dv_, dbeta=dbeta, dlam=dlam, dlog_alpha=dla, d_initial_state=dS0)


def test_three_sweep_backward_equals_oracle_bptt():
    rng = np.random.default_rng(31)
    for T, dk, dv, amean in ((1, 4, 3, 2.0), (23, 6, 5, 2.0), (40, 8, 4, 0.0), (17, 5, 7, 4.0)):
        unit = lambda a: a / np.linalg.norm(a, axis=-1, keepdims=True)
        q, k = unit(rng.standard_normal((T, dk))), unit(rng.standard_normal((T, dk)))
        v = rng.standard_normal((T, dv))
        beta = 1 / (1 + np.exp(-rng.standard_normal(T)))
        lam = 1 / (1 + np.exp(-rng.standard_normal(T)))
        alpha = 1 / (1 + np.exp(-rng.normal(amean, 1.0, T)))
        S0 = 0.3 * rng.standard_normal((dv, dk))
        dO = rng.standard_normal((T, dv))
        dSf = rng.standard_normal((dv, dk))
        got = three_sweep_backward(q, k, v, beta, lam, alpha, S0, dO, dSf)
        sh = lambda a: a[None, :, None]
        ref = recurrent.bwd(q[None, :, None], k[None, :, None], v[None, :, None], sh(beta), sh(lam),
                            np.log(sh(alpha)), S0[None, None], d_o=dO[None, :, None],
                            d_final_state=dSf[None, None])
        for key, val in got.items():
            r = ref[key][0, :, 0] if key != "d_initial_state" else ref[key][0, 0]
            assert np.abs(val - r).max() <= 1e-11 * max(1.0, np.abs(r).max()), (T, key)
