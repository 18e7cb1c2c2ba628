"""fp64 chunkwise form of Q-Delta for any chunk size, forward and backward.

TEST INFRASTRUCTURE ONLY (see the package docstring).  This is not the parity
reference (``recurrent`` is); it checks, in exact-as-possible arithmetic, the
chunk algebra that the GPU kernels follow, so that the kernels can be checked
step by step.

Chunk algebra (Sec. 3.3 "Chunkwise parallel form"; App. D.1 and D.2), for one
chunk of C tokens with entry state S (dv x dk), with the readings that make it
agree with the recurrence (each is pinned by a test):

    b_r   = sum_{j<=r} log alpha_j      (chunk-local prefix sum)
    g_r   = exp(b_r),   Gam_ri = exp(b_r - b_i)
    X     = K + diag(lambda) Q                         (mixed inputs, Eq. (qdelta_gated_form))
    A     = strictLower(diag(beta) (Gam * X K^T))      (row form of the UT transform, App. D.2)
    T     = (I + A)^{-1} diag(beta)
    U     = T V,   W = T diag(g) X                     (one T serves both WY factors)
    D     = U - W S^T                                  ("new values")
    O     = diag(g) Q S^T + (Gam * M * Q K^T) D       (M includes the diagonal)
    S'    = g_C S + D^T diag(g_C / g) K

Readings: the intra-chunk output term carries Gam (the printed chunk output
omits it and is right only for alpha = 1); the query term of the output is
diag(g) Q; the causal mask includes the diagonal; products written "W S" read
as W S^T for S in R^{dv x dk}; App. D.2's "K X^T" reads as X K^T (as in the main
text and the row formula beneath it); the exit-state key weights use row C of
the unmasked Gam.

The backward is the chain rule through exactly these steps (the paper gives
none); it is pinned against the BPTT gradient of ``recurrent``.
"""
import numpy as np


def _chunk_setup(Q, K, V, beta, lam, la):
    n = Q.shape[0]
    b = np.cumsum(la)
    g = np.exp(b)
    Gam = np.exp(b[:, None] - b[None, :])
    X = K + lam[:, None] * Q
    G = X @ K.T
    A = np.tril(beta[:, None] * Gam * G, -1)
    Minv = np.linalg.solve(np.eye(n) + A, np.eye(n))       # (I + A)^{-1}
    T = Minv * beta[None, :]                                 # (I + A)^{-1} diag(beta)
    U = T @ V
    W = T @ (g[:, None] * X)
    QK = Q @ K.T
    mask = np.tril(np.ones((n, n)))                         # inclusive causal mask
    Pm = mask * Gam * QK
    return dict(b=b, g=g, Gam=Gam, X=X, G=G, A=A, Minv=Minv, T=T, U=U, W=W, QK=QK,
                mask=mask, Pm=Pm)


def fwd_unit(q, k, v, beta, lam, log_alpha, S0, C):
    """One (sequence, head): q,k [L,dk], v [L,dv], gates [L], S0 [dv,dk].

    Returns (O [L,dv], S_final, entry_states list)."""
    L = q.shape[0]
    la = np.zeros(L) if log_alpha is None else np.asarray(log_alpha, dtype=np.float64)
    S = np.array(S0, dtype=np.float64, copy=True)
    O = np.zeros((L, v.shape[1]))
    states = []
    for c0 in range(0, L, C):
        sl = slice(c0, min(c0 + C, L))
        st = _chunk_setup(q[sl], k[sl], v[sl], beta[sl], lam[sl], la[sl])
        states.append(S.copy())
        D = st["U"] - st["W"] @ S.T
        O[sl] = st["g"][:, None] * (q[sl] @ S.T) + st["Pm"] @ D
        kb = np.exp(st["b"][-1] - st["b"])
        S = st["g"][-1] * S + D.T @ (kb[:, None] * k[sl])
    return O, S, states


def paper_two_solve_W(k, q, beta, lam, log_alpha):
    """W of Eq. (qdelta_chunk_U) (no decay inside its solve), scaled by diag(g).

    The single-solve W = T diag(g) X used above equals diag(g) times this."""
    n = k.shape[0]
    X = k + lam[:, None] * q
    Wp = np.linalg.solve(np.eye(n) + np.tril(beta[:, None] * (X @ k.T), -1),
                         beta[:, None] * X)
    g = np.exp(np.cumsum(log_alpha))
    return g[:, None] * Wp


def bwd_unit(q, k, v, beta, lam, log_alpha, S0, dO, dSf, C):
    """Gradients of <dO,O> + <dSf,S_T> for one (sequence, head), chunkwise."""
    L, dk = q.shape
    dv = v.shape[1]
    la = np.zeros(L) if log_alpha is None else np.asarray(log_alpha, dtype=np.float64)
    _, _, states = fwd_unit(q, k, v, beta, lam, la, S0, C)
    dq = np.zeros((L, dk)); dkk = np.zeros((L, dk)); dvv = np.zeros((L, dv))
    dbeta = np.zeros(L); dlam = np.zeros(L); dla = np.zeros(L)
    dS = np.zeros((dv, dk)) if dSf is None else np.array(dSf, dtype=np.float64)
    chunks = list(range(0, L, C))
    for ci in reversed(range(len(chunks))):
        c0 = chunks[ci]
        sl = slice(c0, min(c0 + C, L))
        Q, K, V, bt, lm = q[sl], k[sl], v[sl], beta[sl], lam[sl]
        st = _chunk_setup(Q, K, V, bt, lm, la[sl])
        S = states[ci]
        b, g, Gam, X, G = st["b"], st["g"], st["Gam"], st["X"], st["G"]
        T, Minv, U, W, QK, mask, Pm = st["T"], st["Minv"], st["U"], st["W"], st["QK"], st["mask"], st["Pm"]
        gC = g[-1]
        kb = np.exp(b[-1] - b)
        Kbar = kb[:, None] * K
        D = U - W @ S.T
        dOc = dO[sl]
        dSout = dS
        # inter-chunk recursion
        dD = Pm.T @ dOc + Kbar @ dSout.T
        dS = gC * dSout + dOc.T @ (g[:, None] * Q) - dD.T @ W
        # intra-chunk gradients
        db = np.zeros(len(b))
        dOS = dOc @ S
        dQ = g[:, None] * dOS
        db += g * np.sum(Q * dOS, axis=1)
        dPm = mask * (dOc @ D.T)
        dQK = dPm * Gam
        dQ += dQK @ K
        dK = dQK.T @ Q
        dGam = dPm * QK
        dKbar = D @ dSout
        dK += kb[:, None] * dKbar
        t_kb = kb * np.sum(K * dKbar, axis=1)
        db[-1] += t_kb.sum()
        db -= t_kb
        db[-1] += gC * np.sum(dSout * S)
        dU = dD
        dW = -dD @ S
        dV = T.T @ dU
        dT = dU @ V.T + dW @ (g[:, None] * X).T
        dgX = T.T @ dW
        dX = g[:, None] * dgX
        db += g * np.sum(X * dgX, axis=1)
        dbt = np.sum(dT * Minv, axis=0)
        dMinv = dT * bt[None, :]
        dA = np.tril(-Minv.T @ dMinv @ Minv.T, -1)
        dbt += np.sum(dA * Gam * G, axis=1)
        dG = dA * bt[:, None] * Gam
        dGam += dA * bt[:, None] * G
        dX += dG @ K
        dK += dG.T @ X
        dK += dX
        dQ += lm[:, None] * dX
        dlm = np.sum(Q * dX, axis=1)
        rowsum = np.sum(dGam * Gam, axis=1)
        colsum = np.sum(dGam * Gam, axis=0)
        db += rowsum - colsum
        dq[sl] = dQ; dkk[sl] = dK; dvv[sl] = dV
        dbeta[sl] = dbt; dlam[sl] = dlm
        dla[sl] = np.cumsum(db[::-1])[::-1]
    return dict(dq=dq, dk=dkk, dv=dvv, dbeta=dbeta, dlam=dlam,
                dlog_alpha=None if log_alpha is None else dla, d_initial_state=dS)


def _units(q, cu_seqlens):
    if cu_seqlens is None:
        B, T = q.shape[:2]
        return [(b, slice(None)) for b in range(B)], True
    cu = list(cu_seqlens)
    return [(n, slice(cu[n], cu[n + 1])) for n in range(len(cu) - 1)], False


def fwd(q, k, v, beta, lam, log_alpha=None, initial_state=None, C=64, cu_seqlens=None):
    """Chunkwise forward over a batch; same layouts as ``recurrent.fwd``."""
    q, k, v, beta, lam = (np.asarray(a, dtype=np.float64) for a in (q, k, v, beta, lam))
    la = None if log_alpha is None else np.asarray(log_alpha, dtype=np.float64)
    H, dk, dv = q.shape[-2], q.shape[-1], v.shape[-1]
    units, dense = _units(q, cu_seqlens)
    o = np.zeros(v.shape)
    Sf = np.zeros((len(units), H, dv, dk))
    for n, sl in units:
        for h in range(H):
            sel = (n, sl, h) if dense else (sl, h)
            S0 = np.zeros((dv, dk)) if initial_state is None else initial_state[n, h]
            O, S, _ = fwd_unit(q[sel], k[sel], v[sel], beta[sel], lam[sel],
                               None if la is None else la[sel], S0, C)
            o[sel] = O
            Sf[n, h] = S
    return o, Sf


def bwd(q, k, v, beta, lam, log_alpha=None, initial_state=None, d_o=None,
        d_final_state=None, C=64, cu_seqlens=None):
    """Chunkwise backward over a batch; same outputs as ``recurrent.bwd``."""
    q, k, v, beta, lam = (np.asarray(a, dtype=np.float64) for a in (q, k, v, beta, lam))
    la = None if log_alpha is None else np.asarray(log_alpha, dtype=np.float64)
    H, dk, dv = q.shape[-2], q.shape[-1], v.shape[-1]
    units, dense = _units(q, cu_seqlens)
    dO = np.zeros(v.shape) if d_o is None else np.asarray(d_o, dtype=np.float64)
    out = dict(dq=np.zeros(q.shape), dk=np.zeros(k.shape), dv=np.zeros(v.shape),
               dbeta=np.zeros(beta.shape), dlam=np.zeros(lam.shape),
               dlog_alpha=None if la is None else np.zeros(la.shape),
               d_initial_state=np.zeros((len(units), H, dv, dk)))
    for n, sl in units:
        for h in range(H):
            sel = (n, sl, h) if dense else (sl, h)
            S0 = np.zeros((dv, dk)) if initial_state is None else initial_state[n, h]
            dSf = None if d_final_state is None else d_final_state[n, h]
            r = bwd_unit(q[sel], k[sel], v[sel], beta[sel], lam[sel],
                         None if la is None else la[sel], S0, dO[sel], dSf, C)
            for key in ("dq", "dk", "dv", "dbeta", "dlam"):
                out[key][sel] = r[key]
            if la is not None:
                out["dlog_alpha"][sel] = r["dlog_alpha"]
            out["d_initial_state"][n, h] = r["d_initial_state"]
    return out
