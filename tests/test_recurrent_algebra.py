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
