"""Exact rational brute force of the Q-Delta recurrence on tiny inputs.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Two independent evaluations in ``fractions.Fraction`` arithmetic, with no
rounding anywhere:

``dense_product``  the transition-matrix form of Eq. (qdelta_decay):
                   S_t = alpha_t S_{t-1} P_t + beta_t v_t k_t^T with the explicit
                   d_k x d_k matrix P_t = I - beta_t x_t k_t^T, x_t = k_t + lambda_t q_t
                   (Eq. (qdelta_gated_form)).

``closed_form``    the value decomposition of Sec. 3.1 (Eqs. (general_recurrence),
                   (state_decomp), (b_recursion)): the recurrence is the generic
                   S_t = S_{t-1} P'_t + eta_t v_t k_t^T with P'_t = alpha_t P_t and
                   eta_t = beta_t; every state is sum_tau v_tau b_{tau,t}^T with
                   coefficient vectors b_{tau,t} = P'_t^T b_{tau,t-1},
                   b_{t,t} = eta_t k_t.  A non-zero initial state is carried as
                   d_k extra "values" (its columns) whose coefficient vectors start
                   as the unit vectors.  Only vector recursions are used.

Both return (o, S_T) with o_t = S_t q_t.  Inputs are nested lists of numbers
convertible to Fraction.
"""
from fractions import Fraction as Fr


def _F(x):
    return x if isinstance(x, Fr) else Fr(x)


def _vec(a):
    return [_F(x) for x in a]


def _mat(a):
    return [[_F(x) for x in row] for row in a]


def _matmul(A, B):
    n, m, p = len(A), len(B), len(B[0])
    return [[sum((A[i][l] * B[l][j] for l in range(m)), Fr(0)) for j in range(p)] for i in range(n)]


def _matvec(A, x):
    return [sum((a * b for a, b in zip(row, x)), Fr(0)) for row in A]


def dense_product(q, k, v, beta, lam, alpha, S0):
    """q,k: [T][dk]; v: [T][dv]; beta, lam, alpha: [T]; S0: [dv][dk]."""
    T = len(q)
    dk = len(k[0])
    S = _mat(S0)
    o = []
    for t in range(T):
        qt, kt, vt = _vec(q[t]), _vec(k[t]), _vec(v[t])
        bt, lt, at = _F(beta[t]), _F(lam[t]), _F(alpha[t])
        x = [kt[j] + lt * qt[j] for j in range(dk)]
        P = [[(Fr(1) if i == j else Fr(0)) - bt * x[i] * kt[j] for j in range(dk)] for i in range(dk)]
        SP = _matmul(S, P)
        S = [[at * SP[i][j] + bt * vt[i] * kt[j] for j in range(dk)] for i in range(len(S))]
        o.append(_matvec(S, qt))
    return o, S


def closed_form(q, k, v, beta, lam, alpha, S0):
    """Same inputs as ``dense_product``; evaluates the value decomposition."""
    T = len(q)
    dk = len(k[0])
    dv = len(v[0])
    S0 = _mat(S0)
    # "values" and their coefficient vectors: initial-state columns first
    values = [[S0[i][j] for i in range(dv)] for j in range(dk)]
    coefs = [[Fr(1) if l == j else Fr(0) for l in range(dk)] for j in range(dk)]
    o = []
    for t in range(T):
        qt, kt, vt = _vec(q[t]), _vec(k[t]), _vec(v[t])
        bt, lt, at = _F(beta[t]), _F(lam[t]), _F(alpha[t])
        x = [kt[j] + lt * qt[j] for j in range(dk)]
        # b <- P'_t^T b = alpha_t (b - beta_t k_t (x_t . b))
        new = []
        for bvec in coefs:
            xb = sum((x[j] * bvec[j] for j in range(dk)), Fr(0))
            new.append([at * (bvec[j] - bt * kt[j] * xb) for j in range(dk)])
        coefs = new
        values.append(vt)
        coefs.append([bt * kt[j] for j in range(dk)])
        # o_t = S_t q_t = sum_tau v_tau (b_{tau,t} . q_t)
        w = [sum((bvec[j] * qt[j] for j in range(dk)), Fr(0)) for bvec in coefs]
        o.append([sum((values[m][i] * w[m] for m in range(len(values))), Fr(0)) for i in range(dv)])
    S = [[sum((values[m][i] * coefs[m][j] for m in range(len(values))), Fr(0)) for j in range(dk)]
         for i in range(dv)]
    return o, S
