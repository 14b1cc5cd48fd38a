"""CPU fp64 oracle for the gated linear attention (GLA) layer.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this package; the product path
(``paper_2312_06635_amd``) never does, and the two share no code.

``fwd`` / ``bwd`` call the plain C recurrence in ``gla_oracle.c`` (paper,
Sec. 4.1, Eq. 3, and its reverse mode); ``forms`` holds the independent numpy
formulations (chunkwise form of Sec. 4.2 with the secondary chunking of
Sec. 4.3, the log-space parallel form of Eq. 4, and the closed-form gate
gradient) that pin the recurrence.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gla_oracle.c")
_LIB = os.path.join(_HERE, "libgla_oracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile gla_oracle.c with gcc into oracle/libgla_oracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fPIC", "-shared", "-std=c99", "-pthread", "-o", tmp, _SRC, "-lm"]
        )
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        i64 = ctypes.c_int64
        lib.gla_oracle_fwd.argtypes = [i64, i64, i64, i64, dp, dp, dp, dp, dp, dp, dp, ctypes.c_int]
        lib.gla_oracle_fwd.restype = ctypes.c_int
        lib.gla_oracle_bwd.argtypes = [i64, i64, i64, i64, dp, dp, dp, dp, dp, dp, dp,
                                       dp, dp, dp, dp, dp, ctypes.c_int, i64]
        lib.gla_oracle_bwd.restype = ctypes.c_int
        _lib = lib
    return _lib


def _as_f64(x):
    if x is None:
        return None
    if hasattr(x, "detach"):  # torch tensor
        x = x.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(x, dtype=np.float64)


def _ptr(a):
    if a is None:
        return ctypes.POINTER(ctypes.c_double)()
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)))


def fwd(q, k, v, log_alpha, S0=None, want_state=True, nthreads=None):
    """Recurrent forward (Eq. 3) in fp64.

    q, k, log_alpha: [..., T, d_k]; v: [..., T, d_v]; S0: [..., d_k, d_v] or None.
    Leading dims are flattened into independent heads.  Returns (o, S_T) as
    float64 numpy arrays with the input's leading shape (S_T None if not wanted).
    """
    q, k, v, la, S0 = (_as_f64(x) for x in (q, k, v, log_alpha, S0))
    lead = q.shape[:-2]
    T, K = q.shape[-2:]
    V = v.shape[-1]
    BH = int(np.prod(lead)) if lead else 1
    o = np.empty(lead + (T, V), np.float64)
    ST = np.empty(lead + (K, V), np.float64) if want_state else None
    rc = _load().gla_oracle_fwd(BH, T, K, V, _ptr(q), _ptr(k), _ptr(v), _ptr(la), _ptr(S0),
                                _ptr(o), _ptr(ST), nthreads or default_threads())
    if rc != 0:
        raise RuntimeError(f"gla_oracle_fwd failed ({rc})")
    return o, ST


def bwd(q, k, v, log_alpha, dO, S0=None, dST=None, nthreads=None, ckpt=64):
    """Back-propagation through the recurrence of Eq. 3 in fp64.

    Loss convention: L = sum(o * dO) + sum(S_T * dS_T).
    Returns dict with dq, dk, dv, dlog_alpha, dS0 (float64 numpy arrays).
    """
    q, k, v, la, dO, S0, dST = (_as_f64(x) for x in (q, k, v, log_alpha, dO, S0, dST))
    lead = q.shape[:-2]
    T, K = q.shape[-2:]
    V = v.shape[-1]
    BH = int(np.prod(lead)) if lead else 1
    dq = np.empty_like(q)
    dk = np.empty_like(q)
    dla = np.empty_like(q)
    dv = np.empty_like(v)
    dS0 = np.empty(lead + (K, V), np.float64)
    rc = _load().gla_oracle_bwd(BH, T, K, V, _ptr(q), _ptr(k), _ptr(v), _ptr(la), _ptr(S0),
                                _ptr(dO), _ptr(dST), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dla),
                                _ptr(dS0), nthreads or default_threads(), ckpt)
    if rc != 0:
        raise RuntimeError(f"gla_oracle_bwd failed ({rc})")
    return {"dq": dq, "dk": dk, "dv": dv, "dlog_alpha": dla, "dS0": dS0}


def gate_log_alpha(z, tau):
    """log alpha of the GLA gate from its pre-activation z (paper, Sec. 4.4 and
    Table 1): alpha = sigmoid(z)^(1/tau), so log alpha = logsigmoid(z) / tau.
    logsigmoid(z) = -log(1 + exp(-z)) is evaluated as min(z, 0) -
    log1p(exp(-|z|)), which never overflows."""
    z = _as_f64(z)
    return (np.minimum(z, 0.0) - np.log1p(np.exp(-np.abs(z)))) / tau


def gate_grad(z, tau, dlog_alpha):
    """Chain rule through gate_log_alpha: d logsigmoid(z) / dz = sigmoid(-z),
    so dL/dz = dL/dlog_alpha * sigmoid(-z) / tau, with sigmoid(-z) =
    (1 - tanh(z / 2)) / 2."""
    z = _as_f64(z)
    return _as_f64(dlog_alpha) * (0.5 * (1.0 - np.tanh(0.5 * z))) / tau


# ---------------------------------------------------------------- output side
# The GLA Transformer's per-head output (paper, Sec. 4.4): LayerNorm of each
# head's output o_t (affine parameters per channel of the concatenated heads,
# as in the group normalisation of the cited RetNet design) gated by
# r_t = Swish(g_t), g_t the output-gate pre-activation (its projection is a
# plain GEMM outside this layer): y_t = r_t (.) LN(o_t).

def _sigmoid(x):
    return 0.5 * (1.0 + np.tanh(0.5 * x))


def output_gate_fwd(o, g, w=None, b=None, eps=1e-5):
    """o, g: [..., H, T, d_v] (per-head rows); w, b: [H, d_v] or None (1 / 0).
    Returns (y, mean, rstd) with mean and rstd = 1/sqrt(var + eps) per row."""
    o, g = _as_f64(o), _as_f64(g)
    mu = o.mean(axis=-1, keepdims=True)
    var = ((o - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xh = (o - mu) * rstd
    H = o.shape[-3]
    wv = np.ones((H, o.shape[-1])) if w is None else _as_f64(w)
    bv = np.zeros((H, o.shape[-1])) if b is None else _as_f64(b)
    ln = xh * wv[:, None, :] + bv[:, None, :]
    r = g * _sigmoid(g)
    return r * ln, mu[..., 0], rstd[..., 0]


def output_gate_bwd(o, g, dy, w=None, b=None, eps=1e-5):
    """Reverse mode of output_gate_fwd for L = sum(y * dy).
    Returns dict(do, dg, dw, db); dw, db are [H, d_v]."""
    o, g, dy = _as_f64(o), _as_f64(g), _as_f64(dy)
    H, V = o.shape[-3], o.shape[-1]
    wv = np.ones((H, V)) if w is None else _as_f64(w)
    bv = np.zeros((H, V)) if b is None else _as_f64(b)
    mu = o.mean(axis=-1, keepdims=True)
    var = ((o - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xh = (o - mu) * rstd
    ln = xh * wv[:, None, :] + bv[:, None, :]
    s = _sigmoid(g)
    r = g * s
    dg = dy * ln * (s * (1.0 + g * (1.0 - s)))       # d swish(g)/dg = s (1 + g (1 - s))
    dln = dy * r
    lead = tuple(range(o.ndim - 3))
    dw = (dln * xh).sum(axis=lead + (o.ndim - 2,))
    db = dln.sum(axis=lead + (o.ndim - 2,))
    dxh = dln * wv[:, None, :]
    do = rstd * (dxh - dxh.mean(axis=-1, keepdims=True) - xh * (dxh * xh).mean(axis=-1, keepdims=True))
    return {"do": do, "dg": dg, "dw": dw, "db": db}


# ---------------------------------------------------------------- scalar gates
# Data-dependent scalar gates (Table 1: the Mamba-2, mLSTM and Gated Retention
# rows, G_t = gamma_t 1^T 1): one decay per step and head, shared by every key
# feature.  As a GLA layer this is alpha_t = gamma_t 1 (Sec. 4.1, Eq. 3), and
# by the chain rule of that broadcast dL/dlog gamma_t = sum over the key
# features of dL/dlog alpha_t.

def _broadcast_gate(log_gamma, K):
    lg = _as_f64(log_gamma)
    return np.ascontiguousarray(np.broadcast_to(lg[..., None], lg.shape + (K,)))


def scalar_gate_fwd(q, k, v, log_gamma, S0=None, want_state=True, nthreads=None):
    """Forward recurrence with G_t = gamma_t 1^T 1; log_gamma: [..., T]."""
    K = _as_f64(q).shape[-1]
    return fwd(q, k, v, _broadcast_gate(log_gamma, K), S0, want_state=want_state, nthreads=nthreads)


def scalar_gate_bwd(q, k, v, log_gamma, dO, S0=None, dST=None, nthreads=None, ckpt=64):
    """Reverse mode of scalar_gate_fwd; returns dq, dk, dv, dS0 and
    dlog_gamma ([..., T])."""
    K = _as_f64(q).shape[-1]
    g = bwd(q, k, v, _broadcast_gate(log_gamma, K), dO, S0=S0, dST=dST, nthreads=nthreads, ckpt=ckpt)
    g["dlog_gamma"] = g.pop("dlog_alpha").sum(axis=-1)
    return g


# ---------------------------------------------------------------- general gates
# The general gated form of App. C: G_t = alpha_t^T beta_t, a key-side gate
# alpha_t in (0,1]^{d_k} and a value-side gate beta_t in (0,1]^{d_v},
#     S_t = (alpha_t^T beta_t) (.) S_{t-1} + k_t^T v_t,    o_t = q_t S_t.
# Plain numpy, one step at a time (all leading dims at once), fp64.

def general_gate_fwd(q, k, v, log_alpha, log_beta, S0=None):
    """Returns (o, S_T); q, k, log_alpha: [..., T, d_k]; v, log_beta:
    [..., T, d_v]; S0: [..., d_k, d_v] or None."""
    q, k, v, la, lb, S0 = (_as_f64(x) for x in (q, k, v, log_alpha, log_beta, S0))
    T, K = q.shape[-2:]
    V = v.shape[-1]
    S = np.zeros(q.shape[:-2] + (K, V)) if S0 is None else S0.copy()
    o = np.empty(q.shape[:-1] + (V,))
    for t in range(T):
        S = np.exp(la[..., t, :, None] + lb[..., t, None, :]) * S + k[..., t, :, None] * v[..., t, None, :]
        o[..., t, :] = np.einsum("...a,...aj->...j", q[..., t, :], S)
    return o, S


def general_gate_bwd(q, k, v, log_alpha, log_beta, dO, S0=None, dST=None, ckpt=64):
    """Back-propagation through general_gate_fwd for L = sum(o dO) +
    sum(S_T dS_T).  With G_t = dL/dS_t and M_t = alpha_t^T beta_t:
    G_t = q_t^T do_t + M_{t+1} (.) G_{t+1} (G_T also holds dS_T),
    dq_t = S_t do_t^T, dk_t = G_t v_t^T, dv_t = k_t G_t,
    d log alpha_t = rowsum(G_t (.) M_t (.) S_{t-1}), d log beta_t the column
    sums of the same product, dS0 = M_1 (.) G_1.  States are kept every ckpt
    steps and recomputed segment by segment.  Returns dq, dk, dv, dlog_alpha,
    dlog_beta, dS0."""
    q, k, v, la, lb, dO, S0, dST = (_as_f64(x) for x in (q, k, v, log_alpha, log_beta, dO, S0, dST))
    T, K = q.shape[-2:]
    V = v.shape[-1]
    lead = q.shape[:-2]
    M = lambda t: np.exp(la[..., t, :, None] + lb[..., t, None, :])
    step = lambda S, t: M(t) * S + k[..., t, :, None] * v[..., t, None, :]
    S = np.zeros(lead + (K, V)) if S0 is None else S0.copy()
    ck = {0: S}
    for t in range(T):
        S = step(S, t)
        if (t + 1) % ckpt == 0:
            ck[t + 1] = S
    G = np.zeros(lead + (K, V)) if dST is None else dST.copy()
    out = {n: np.zeros_like(x) for n, x in (("dq", q), ("dk", k), ("dv", v), ("dlog_alpha", la),
                                               ("dlog_beta", lb))}
    for s0 in range(((T - 1) // ckpt) * ckpt if T else 0, -1, -ckpt):
        seg = [ck[s0]]  # seg[i] = S_{s0 + i}
        for t in range(s0, min(s0 + ckpt, T)):
            seg.append(step(seg[-1], t))
        for t in range(min(s0 + ckpt, T) - 1, s0 - 1, -1):
            Sp, Sc, Mt = seg[t - s0], seg[t - s0 + 1], M(t)
            G = G + q[..., t, :, None] * dO[..., t, None, :]
            out["dq"][..., t, :] = np.einsum("...aj,...j->...a", Sc, dO[..., t, :])
            out["dk"][..., t, :] = np.einsum("...aj,...j->...a", G, v[..., t, :])
            out["dv"][..., t, :] = np.einsum("...a,...aj->...j", k[..., t, :], G)
            dM = G * Mt * Sp
            out["dlog_alpha"][..., t, :] = dM.sum(axis=-1)
            out["dlog_beta"][..., t, :] = dM.sum(axis=-2)
            G = Mt * G
    out["dS0"] = G
    return out
