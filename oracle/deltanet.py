"""DeltaNet and GatedDeltaNet rules, written out on their own.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 2.1, Eq. (delta_rule):  S_t = S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
Sec. 2.1, Eq. (gated_delta_recurrence):
                             S_t = S_{t-1} (alpha_t (I - beta_t k_t k_t^T)) + beta_t v_t k_t^T
with read-out o_t = S_t q_t.  Q-Delta with lambda = 0 must reduce to these.
"""
import numpy as np


def gated_delta(q, k, v, beta, alpha, S0):
    """One sequence and head: q,k [T,dk], v [T,dv], beta/alpha [T] (alpha None = 1)."""
    S = np.array(S0, dtype=np.float64, copy=True)
    I = np.eye(k.shape[1])
    o = np.zeros((q.shape[0], v.shape[1]))
    for t in range(q.shape[0]):
        a = 1.0 if alpha is None else alpha[t]
        S = S @ (a * (I - beta[t] * np.outer(k[t], k[t]))) + beta[t] * np.outer(v[t], k[t])
        o[t] = S @ q[t]
    return o, S
