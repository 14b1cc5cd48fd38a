"""Independent fp64 numpy formulations of the GLA layer, used to pin the oracle.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).  Every function works
on a single head: q, k, log_alpha are [T, d_k], v and dO are [T, d_v], states
are [d_k, d_v].  None of this is shared with the HIP library.
"""
from __future__ import annotations

import numpy as np


def _f64(x):
    if x is None:
        return None
    if hasattr(x, "detach"):
        x = x.detach().to("cpu").double().numpy()
    return np.asarray(x, dtype=np.float64)


def causal_linear_attention(q, k, v, S0=None):
    """Ungated causal linear attention, parallel form O = ((Q K^T) (.) M) V (Sec. 2.1),
    where M_ij = 1 iff i >= j; an initial state adds Q S0 (Sec. 2.2)."""
    q, k, v, S0 = map(_f64, (q, k, v, S0))
    T = q.shape[0]
    M = np.tril(np.ones((T, T)))
    o = ((q @ k.T) * M) @ v
    if S0 is not None:
        o = o + q @ S0
    return o


def decay_mask_attention(q, k, v, gamma):
    """Constant scalar decay gamma (the RetNet special case named in Sec. 4 and
    App. C): O = ((Q K^T) (.) D) V with D_ij = gamma^(i-j) for i >= j, else 0."""
    q, k, v = map(_f64, (q, k, v))
    T = q.shape[0]
    i = np.arange(T)[:, None]
    j = np.arange(T)[None, :]
    D = np.where(i >= j, float(gamma) ** np.maximum(i - j, 0), 0.0)
    return ((q @ k.T) * D) @ v


def parallel_logspace(q, k, v, log_alpha, S0=None):
    """Log-space parallel form of GLA (Sec. 4.1, Eq. 4):
    P_ij = sum_k Q_ik K_jk exp(log B_ik - log B_jk) for i >= j, O = P V, where
    log B_t = sum_{s <= t} log alpha_s.  An initial state adds (Q (.) B) S0."""
    q, k, v, la, S0 = map(_f64, (q, k, v, log_alpha, S0))
    T = q.shape[0]
    logB = np.cumsum(la, axis=0)
    mask = np.tril(np.ones((T, T), bool))
    diff = np.where(mask[:, :, None], logB[:, None, :] - logB[None, :, :], -np.inf)
    P = np.einsum("ik,jk,ijk->ij", q, k, np.exp(diff))
    o = P @ v
    if S0 is not None:
        o = o + (q * np.exp(logB)) @ S0
    return o


def _chunk_factors(la_c):
    """Chunk-local inclusive cumsum of log gates and the decay factors of Sec. 4.2:
    B[j] = log(b_{iC+j+1} / b_{iC}); Lambda = exp(B); Gamma = exp(B_last - B);
    gamma = exp(B_last)."""
    B = np.cumsum(la_c, axis=0)
    Bl = B[-1]
    return B, Bl, np.exp(B), np.exp(Bl - B), np.exp(Bl)


def chunk_fwd(q, k, v, log_alpha, C, c, S0=None):
    """Chunkwise form of GLA (Sec. 4.2) with secondary chunking (Sec. 4.3).

    Inter-chunk:  O_inter = (Q (.) Lambda) S_[n];
                  S_[n+1] = (gamma^T 1) (.) S_[n] + (K (.) Gamma)^T V.
    Intra-chunk, sub-chunks of length c: a sub-chunk against itself in log space
    (Eq. 4, the pink tiles of Fig. 3); a sub-chunk i against an earlier one j by
    a plain product of normalized operands (the orange tiles): the normalizer is
    log b at the boundary just before sub-chunk i, so every exponent is <= 0.
    Returns (O [T, d_v], S_T [d_k, d_v])."""
    q, k, v, la, S0 = map(_f64, (q, k, v, log_alpha, S0))
    T, K = q.shape
    V = v.shape[1]
    assert T % C == 0 and C % c == 0
    S = np.zeros((K, V)) if S0 is None else S0.copy()
    O = np.zeros((T, V))
    tri = np.tril(np.ones((c, c), bool))[:, :, None]
    for n in range(T // C):
        r = slice(n * C, (n + 1) * C)
        qc, kc, vc = q[r], k[r], v[r]
        B, Bl, Lam, Gam, gam = _chunk_factors(la[r])
        Oc = (qc * Lam) @ S
        for i in range(C // c):
            ri = slice(i * c, (i + 1) * c)
            Bi = B[ri]
            W = np.exp(np.where(tri, Bi[:, None, :] - Bi[None, :, :], -np.inf))
            P = np.einsum("mk,nk,mnk->mn", qc[ri], kc[ri], W)
            Oc[ri] += P @ vc[ri]
            if i > 0:
                z = B[i * c - 1]
                qn = qc[ri] * np.exp(Bi - z)
                for j in range(i):
                    rj = slice(j * c, (j + 1) * c)
                    kn = kc[rj] * np.exp(z - B[rj])
                    Oc[ri] += (qn @ kn.T) @ vc[rj]
        O[r] = Oc
        S = gam[:, None] * S + (kc * Gam).T @ vc
    return O, S


def dlog_alpha_closed_form(q, k, dq, dk, ST=None, dST=None):
    """Closed-form gate gradient (Sec. 4.3, derived in App. B):
    dlog b_t = q_t (.) dq_t - k_t (.) dk_t and dlog alpha_t = sum_{i >= t} dlog b_i.
    When a gradient dS_T flows into the final state, log b_T also reaches the
    loss through S_T = Diag(b_T)(...), which adds rowsum(S_T (.) dS_T) to every t."""
    q, k, dq, dk, ST, dST = map(_f64, (q, k, dq, dk, ST, dST))
    dA = q * dq - k * dk
    out = np.flip(np.cumsum(np.flip(dA, 0), 0), 0).copy()
    if ST is not None and dST is not None:
        out += (ST * dST).sum(axis=1)[None, :]
    return out


def chunk_bwd(q, k, v, log_alpha, dO, C, c, S0=None, dST=None):
    """Backward of the chunkwise form (the structure of App. B, Alg. 4, with its
    typos corrected: the reverse state pass uses Q (.) Lambda, and the intra
    gradients use the same secondary chunking as the forward).

    States S_[n] are recomputed by a forward pass; the reverse pass carries
    dS = dL/dS_[n+1]:  dS_[n] = (gamma^T 1) (.) dS + (Q (.) Lambda)^T dO_[n].
    Loss convention: L = sum(O * dO) + sum(S_T * dS_T).
    Returns dict(dq, dk, dv, dlog_alpha, dS0)."""
    q, k, v, la, dO, S0, dST = map(_f64, (q, k, v, log_alpha, dO, S0, dST))
    T, K = q.shape
    V = v.shape[1]
    N = T // C
    assert T % C == 0 and C % c == 0
    S = np.zeros((K, V)) if S0 is None else S0.copy()
    states = []
    for n in range(N):
        states.append(S)
        r = slice(n * C, (n + 1) * C)
        B, Bl, Lam, Gam, gam = _chunk_factors(la[r])
        S = gam[:, None] * S + (k[r] * Gam).T @ v[r]
    ST = S
    dS = np.zeros((K, V)) if dST is None else dST.copy()
    dq = np.zeros_like(q)
    dk = np.zeros_like(q)
    dv = np.zeros_like(v)
    tri2 = np.tril(np.ones((c, c)))
    tri = tri2.astype(bool)[:, :, None]
    for n in reversed(range(N)):
        r = slice(n * C, (n + 1) * C)
        qc, kc, vc, dOc = q[r], k[r], v[r], dO[r]
        B, Bl, Lam, Gam, gam = _chunk_factors(la[r])
        dqc = (dOc @ states[n].T) * Lam
        dkc = (vc @ dS.T) * Gam
        dvc = (kc * Gam) @ dS
        for i in range(C // c):
            ri = slice(i * c, (i + 1) * c)
            Bi = B[ri]
            W = np.exp(np.where(tri, Bi[:, None, :] - Bi[None, :, :], -np.inf))
            P = np.einsum("mk,nk,mnk->mn", qc[ri], kc[ri], W)
            dP = (dOc[ri] @ vc[ri].T) * tri2
            dqc[ri] += np.einsum("mn,nk,mnk->mk", dP, kc[ri], W)
            dkc[ri] += np.einsum("mn,mk,mnk->nk", dP, qc[ri], W)
            dvc[ri] += P.T @ dOc[ri]
            if i > 0:
                z = B[i * c - 1]
                eq = np.exp(Bi - z)
                qn = qc[ri] * eq
                for j in range(i):
                    rj = slice(j * c, (j + 1) * c)
                    ek = np.exp(z - B[rj])
                    kn = kc[rj] * ek
                    dPij = dOc[ri] @ vc[rj].T
                    dqc[ri] += (dPij @ kn) * eq
                    dkc[rj] += (dPij.T @ qn) * ek
                    dvc[rj] += (qn @ kn.T).T @ dOc[ri]
        dq[r], dk[r], dv[r] = dqc, dkc, dvc
        dS = gam[:, None] * dS + (qc * Lam).T @ dOc
    dla = dlog_alpha_closed_form(q, k, dq, dk, ST, dST)
    return {"dq": dq, "dk": dk, "dv": dv, "dlog_alpha": dla, "dS0": dS}


def scalar_decay_attention(q, k, v, log_gamma, S0=None):
    """Parallel form of linear attention with a data-dependent scalar decay
    (the scalar-gate rows of Table 1, G_t = gamma_t 1^T 1): with
    c_t = sum_{s <= t} log gamma_s, O = ((Q K^T) (.) D) V, D_ij = exp(c_i - c_j)
    for i >= j, else 0; an initial state adds exp(c_i) q_i S0.  Also returns
    the final state S_T = sum_s exp(c_T - c_s) k_s^T v_s + exp(c_T) S0."""
    q, k, v, lg, S0 = map(_f64, (q, k, v, log_gamma, S0))
    T = q.shape[0]
    c = np.cumsum(lg)
    i = np.arange(T)[:, None]
    j = np.arange(T)[None, :]
    D = np.where(i >= j, np.exp(np.where(i >= j, c[:, None] - c[None, :], 0.0)), 0.0)
    o = ((q @ k.T) * D) @ v
    cT = c[-1] if T else 0.0
    ST = (k * np.exp(cT - c)[:, None]).T @ v
    if S0 is not None:
        o = o + np.exp(c)[:, None] * (q @ S0)
        ST = ST + np.exp(cT) * S0
    return o, ST


def general_gate_parallel(q, k, v, log_alpha, log_beta, S0=None):
    """Parallel form of the general gate G_t = alpha_t^T beta_t (App. C): with
    A, D the cumulative sums of log alpha and log beta,
    o_t[j] = sum_{s <= t} sum_a q_t[a] k_s[a] v_s[j] exp(A_t[a] - A_s[a] + D_t[j] - D_s[j])
             + sum_a q_t[a] exp(A_t[a] + D_t[j]) S0[a, j]."""
    q, k, v, la, lb, S0 = map(_f64, (q, k, v, log_alpha, log_beta, S0))
    T = q.shape[0]
    A, D = np.cumsum(la, axis=0), np.cumsum(lb, axis=0)
    mask = np.tril(np.ones((T, T), bool))
    ea = np.where(mask[:, :, None], np.exp(np.where(mask[:, :, None], A[:, None, :] - A[None, :, :], 0.0)), 0.0)
    ed = np.where(mask[:, :, None], np.exp(np.where(mask[:, :, None], D[:, None, :] - D[None, :, :], 0.0)), 0.0)
    o = np.einsum("ta,sa,tsa,sj,tsj->tj", q, k, ea, v, ed)
    if S0 is not None:
        o = o + np.einsum("ta,ta,aj,tj->tj", q, np.exp(A), S0, np.exp(D))
    return o


def general_gate_closed_form(q, k, v, o, dq, dk, dv, dO, ST=None, dST=None):
    """Gate gradients of the general form without the states (App. C):
    dlog alpha_t = sum_{i >= t} (q_i dq_i - k_i dk_i) + rowsum(S_T dS_T) and,
    on the value side, dlog beta_t = sum_{i >= t} (o_i do_i - v_i dv_i)
    + colsum(S_T dS_T)."""
    q, k, v, o, dq, dk, dv, dO, ST, dST = map(_f64, (q, k, v, o, dq, dk, dv, dO, ST, dST))
    ra = np.cumsum((q * dq - k * dk)[::-1], axis=0)[::-1]
    rb = np.cumsum((o * dO - v * dv)[::-1], axis=0)[::-1]
    if ST is not None and dST is not None:
        ra = ra + (ST * dST).sum(axis=1)[None, :]
        rb = rb + (ST * dST).sum(axis=0)[None, :]
    return ra, rb
