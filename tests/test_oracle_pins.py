"""Pins of the fp64 CPU oracle against what the paper and the mathematics fix.

The oracle (plain recurrence of Sec. 4.1, Eq. 3 and its reverse mode) is checked
against hand-derived worked examples, textbook closed forms (ungated causal
linear attention, constant decay), the log-space parallel form (Eq. 4), an
independent chunkwise reimplementation (Sec. 4.2/4.3), central finite
differences, the closed-form gate gradient, and invariants (causality,
linearity, segment split, vanishing gate).  CPU only.
"""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import forms

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.abs(a - b).max() / max(np.abs(b).max(), 1e-300)


def rand_case(rng, T, K, V, gate_scale=1.0, with_s0=False):
    q = rng.standard_normal((T, K))
    k = rng.standard_normal((T, K)) / np.sqrt(K)
    v = rng.standard_normal((T, V))
    x = rng.standard_normal((T, K))
    la = -np.logaddexp(0.0, -x) * gate_scale       # log sigmoid(x), <= 0
    S0 = rng.standard_normal((K, V)) * 0.3 if with_s0 else None
    return q, k, v, la, S0


# ---------------------------------------------------------------- worked examples

def test_golden_scalar_recurrence_and_gradient():
    g = json.load(open(os.path.join(GOLDEN, "scalar_T3.json")))
    col = lambda x: np.asarray(x, np.float64).reshape(-1, 1)
    q, k, v = col(g["q"]), col(g["k"]), col(g["v"])
    la = np.log(col(g["alpha"]))
    S0 = np.array([[g["S0"]]])
    o, ST = oracle.fwd(q, k, v, la, S0)
    assert np.allclose(o[:, 0], g["o"], rtol=1e-14, atol=0)
    assert np.isclose(ST[0, 0], g["S_T"], rtol=1e-14)
    gr = oracle.bwd(q, k, v, la, col(g["dO"]), S0=S0)
    for name in ("dq", "dk", "dv", "dlog_alpha"):
        assert np.allclose(gr[name][:, 0], g[name], rtol=1e-13, atol=1e-15), name
    assert np.isclose(gr["dS0"][0, 0], g["dS0"], rtol=1e-14)


def test_golden_gate_acts_on_key_rows():
    g = json.load(open(os.path.join(GOLDEN, "diag_gate_K2.json")))
    a = lambda x: np.asarray(x, np.float64)
    o, ST = oracle.fwd(a(g["q"]), a(g["k"]), a(g["v"]), np.log(a(g["alpha"])))
    assert np.allclose(o, a(g["o"]), rtol=1e-14)
    assert np.allclose(ST, a(g["S_T"]), rtol=1e-14)


# ---------------------------------------------------------------- closed forms

def test_ungated_equals_causal_linear_attention():
    rng = np.random.default_rng(1)
    q, k, v, _, S0 = rand_case(rng, 37, 5, 7, with_s0=True)
    la = np.zeros_like(q)
    o, ST = oracle.fwd(q, k, v, la, S0)
    assert rel(o, forms.causal_linear_attention(q, k, v, S0)) < 1e-12
    assert rel(ST, S0 + k.T @ v) < 1e-12


def test_constant_decay_equals_decay_mask():
    rng = np.random.default_rng(2)
    q, k, v, _, _ = rand_case(rng, 41, 6, 4)
    gamma = 0.87
    la = np.full_like(q, np.log(gamma))
    o, _ = oracle.fwd(q, k, v, la)
    assert rel(o, forms.decay_mask_attention(q, k, v, gamma)) < 1e-12


@pytest.mark.parametrize("gate_scale", [1 / 16, 1.0, 6.0])
def test_recurrence_equals_logspace_parallel_form(gate_scale):
    rng = np.random.default_rng(3)
    q, k, v, la, S0 = rand_case(rng, 29, 6, 5, gate_scale=gate_scale, with_s0=True)
    o, _ = oracle.fwd(q, k, v, la, S0)
    assert rel(o, forms.parallel_logspace(q, k, v, la, S0)) < 1e-12


def test_vanishing_gate_keeps_only_the_diagonal():
    rng = np.random.default_rng(4)
    q, k, v, _, S0 = rand_case(rng, 19, 4, 3, with_s0=True)
    la = np.full_like(q, -50.0)
    o, _ = oracle.fwd(q, k, v, la, S0)
    ref = (q * k).sum(1, keepdims=True) * v
    assert rel(o, ref) < 1e-12


# ---------------------------------------------------------------- chunk form

@pytest.mark.parametrize("C,c", [(1, 1), (4, 2), (8, 8), (16, 8), (16, 4), (48, 16), (48, 48),
                                 (6, 3)])
def test_recurrence_equals_chunk_form(C, c):
    rng = np.random.default_rng(5)
    T = 48
    q, k, v, la, S0 = rand_case(rng, T, 6, 5, gate_scale=1 / 16, with_s0=True)
    o, ST = oracle.fwd(q, k, v, la, S0)
    oc, STc = forms.chunk_fwd(q, k, v, la, C, c, S0)
    assert rel(o, oc) < 1e-12
    assert rel(ST, STc) < 1e-12


def test_chunk_form_strong_decay_stays_finite():
    rng = np.random.default_rng(6)
    q, k, v, _, _ = rand_case(rng, 32, 4, 3)
    la = -rng.uniform(5, 40, size=q.shape)
    o, _ = oracle.fwd(q, k, v, la)
    oc, _ = forms.chunk_fwd(q, k, v, la, 16, 4)
    assert np.isfinite(oc).all()
    assert rel(o, oc) < 1e-12


# ---------------------------------------------------------------- gradients

def _loss(q, k, v, la, S0, dO, dST):
    o, ST = oracle.fwd(q, k, v, la, S0, nthreads=1)
    return (o * dO).sum() + (ST * dST).sum()


def test_gradients_match_central_finite_differences():
    rng = np.random.default_rng(7)
    T, K, V = 6, 3, 2
    q, k, v, la, S0 = rand_case(rng, T, K, V, gate_scale=0.5, with_s0=True)
    dO = rng.standard_normal((T, V))
    dST = rng.standard_normal((K, V))
    g = oracle.bwd(q, k, v, la, dO, S0=S0, dST=dST, nthreads=1, ckpt=4)
    args = {"q": q, "k": k, "v": v, "la": la, "S0": S0}
    grads = {"q": g["dq"], "k": g["dk"], "v": g["dv"], "la": g["dlog_alpha"], "S0": g["dS0"]}
    h = 1e-6
    for name, x in args.items():
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp = x.copy(); xp[idx] += h
            xm = x.copy(); xm[idx] -= h
            ap = dict(args); ap[name] = xp
            am = dict(args); am[name] = xm
            fd[idx] = (_loss(ap["q"], ap["k"], ap["v"], ap["la"], ap["S0"], dO, dST)
                       - _loss(am["q"], am["k"], am["v"], am["la"], am["S0"], dO, dST)) / (2 * h)
        assert rel(grads[name], fd) < 1e-7, name


@pytest.mark.parametrize("with_state", [False, True])
def test_bptt_equals_chunk_form_backward(with_state):
    rng = np.random.default_rng(8)
    T, K, V = 64, 8, 6
    q, k, v, la, S0 = rand_case(rng, T, K, V, gate_scale=1 / 4, with_s0=with_state)
    dO = rng.standard_normal((T, V))
    dST = rng.standard_normal((K, V)) if with_state else None
    g = oracle.bwd(q, k, v, la, dO, S0=S0, dST=dST, ckpt=7)
    gc = forms.chunk_bwd(q, k, v, la, dO, 16, 4, S0=S0, dST=dST)
    for name in ("dq", "dk", "dv", "dlog_alpha", "dS0"):
        assert rel(g[name], gc[name]) < 1e-11, name


def test_direct_gate_gradient_equals_closed_form():
    """Mao et al.'s direct formula (what O2 computes) equals the closed form of
    Sec. 4.3 with the sign q (.) dq - k (.) dk; the opposite sign fails."""
    rng = np.random.default_rng(9)
    T, K, V = 40, 5, 4
    q, k, v, la, _ = rand_case(rng, T, K, V, gate_scale=0.3)
    dO = rng.standard_normal((T, V))
    g = oracle.bwd(q, k, v, la, dO)
    cf = forms.dlog_alpha_closed_form(q, k, g["dq"], g["dk"])
    assert rel(g["dlog_alpha"], cf) < 1e-11
    flipped = np.flip(np.cumsum(np.flip(k * g["dk"] - q * g["dq"], 0), 0), 0)
    assert rel(g["dlog_alpha"], flipped) > 0.1


def test_ungated_gradients_equal_parallel_form_gradients():
    """With alpha = 1 and S0 = 0 the backward of FlashLinearAttention with one
    chunk (App. B, Alg. 2, C = L): dQ = (dO V^T (.) M) K, dK = (V dO^T (.) M^T) Q,
    dV = (Q K^T (.) M)^T dO."""
    rng = np.random.default_rng(10)
    T, K, V = 23, 4, 6
    q, k, v, _, _ = rand_case(rng, T, K, V)
    dO = rng.standard_normal((T, V))
    g = oracle.bwd(q, k, v, np.zeros_like(q), dO)
    M = np.tril(np.ones((T, T)))
    assert rel(g["dq"], ((dO @ v.T) * M) @ k) < 1e-12
    assert rel(g["dk"], ((v @ dO.T) * M.T) @ q) < 1e-12
    assert rel(g["dv"], ((q @ k.T) * M).T @ dO) < 1e-12


# ---------------------------------------------------------------- invariants

def test_causality():
    rng = np.random.default_rng(11)
    q, k, v, la, S0 = rand_case(rng, 30, 4, 3, with_s0=True)
    o, _ = oracle.fwd(q, k, v, la, S0)
    t = 17
    q2, k2, v2, la2 = (x.copy() for x in (q, k, v, la))
    for x in (q2, k2, v2):
        x[t + 1:] += rng.standard_normal(x[t + 1:].shape)
    la2[t + 1:] -= 1.0
    o2, _ = oracle.fwd(q2, k2, v2, la2, S0)
    assert np.array_equal(o[: t + 1], o2[: t + 1])
    assert not np.allclose(o[t + 1:], o2[t + 1:])


def test_linearity_in_v():
    rng = np.random.default_rng(12)
    q, k, v, la, _ = rand_case(rng, 25, 4, 5)
    v2 = rng.standard_normal(v.shape)
    o1, _ = oracle.fwd(q, k, v, la)
    o2, _ = oracle.fwd(q, k, v2, la)
    o3, _ = oracle.fwd(q, k, 2.0 * v - 3.0 * v2, la)
    assert rel(o3, 2.0 * o1 - 3.0 * o2) < 1e-12


def test_segment_split_carries_state():
    rng = np.random.default_rng(13)
    q, k, v, la, S0 = rand_case(rng, 50, 5, 4, with_s0=True)
    o, ST = oracle.fwd(q, k, v, la, S0)
    oa, Sa = oracle.fwd(q[:21], k[:21], v[:21], la[:21], S0)
    ob, Sb = oracle.fwd(q[21:], k[21:], v[21:], la[21:], Sa)
    assert rel(np.concatenate([oa, ob]), o) < 1e-13
    assert rel(Sb, ST) < 1e-13


def test_batched_heads_threads_and_checkpoints_are_consistent():
    rng = np.random.default_rng(14)
    BH, T, K, V = 5, 33, 4, 6
    q = rng.standard_normal((BH, T, K))
    k = rng.standard_normal((BH, T, K))
    v = rng.standard_normal((BH, T, V))
    la = -rng.uniform(0, 0.3, (BH, T, K))
    dO = rng.standard_normal((BH, T, V))
    o1, S1 = oracle.fwd(q, k, v, la, nthreads=1)
    o8, S8 = oracle.fwd(q, k, v, la, nthreads=8)
    assert np.array_equal(o1, o8) and np.array_equal(S1, S8)
    for h in range(BH):
        oh, _ = oracle.fwd(q[h], k[h], v[h], la[h])
        assert np.array_equal(oh, o1[h])
    g1 = oracle.bwd(q, k, v, la, dO, nthreads=1, ckpt=1)
    g2 = oracle.bwd(q, k, v, la, dO, nthreads=8, ckpt=64)
    for name in g1:
        assert np.array_equal(g1[name], g2[name]), name


def test_empty_sequence():
    q = np.zeros((0, 3)); v = np.zeros((0, 2))
    S0 = np.ones((3, 2))
    o, ST = oracle.fwd(q, q, v, q, S0)
    assert o.shape == (0, 2) and np.array_equal(ST, S0)
    g = oracle.bwd(q, q, v, q, v, S0=S0, dST=np.full((3, 2), 2.0))
    assert np.array_equal(g["dS0"], np.full((3, 2), 2.0))


# ---------------------------------------------------------------- gate epilogue

TAU = 16.0  # the temperature the paper fixes for the gate (Sec. 4.4)


def test_gate_epilogue_closed_forms():
    # logsigmoid(0) = -log 2; logsigmoid(z) - logsigmoid(-z) = z exactly
    assert abs(oracle.gate_log_alpha(np.array([0.0]), TAU)[0] + np.log(2.0) / TAU) < 1e-16
    z = np.linspace(-60.0, 60.0, 1201)
    d = oracle.gate_log_alpha(z, 1.0) - oracle.gate_log_alpha(-z, 1.0)
    assert np.abs(d - z).max() < 1e-12
    # alpha = sigmoid(z)^(1/tau) where the direct formula is safe
    zm = np.linspace(-20.0, 20.0, 401)
    alpha = (1.0 / (1.0 + np.exp(-zm))) ** (1.0 / TAU)
    assert rel(np.exp(oracle.gate_log_alpha(zm, TAU)), alpha) < 1e-14
    # tails: log alpha -> -exp(-z)/tau for large z and -> z/tau for very negative z
    big = np.array([30.0, 40.0, 50.0])
    assert rel(oracle.gate_log_alpha(big, TAU), -np.exp(-big) / TAU) < 1e-10
    neg = np.array([-40.0, -50.0])
    assert rel(oracle.gate_log_alpha(neg, TAU), neg / TAU) < 1e-15
    assert np.all(oracle.gate_log_alpha(z, TAU) <= 0.0)


def test_gate_gradient_matches_central_finite_differences():
    z = np.linspace(-12.0, 12.0, 97)
    g = np.linspace(-1.0, 2.0, 97)
    h = 1e-5
    fd = g * (oracle.gate_log_alpha(z + h, TAU) - oracle.gate_log_alpha(z - h, TAU)) / (2 * h)
    assert rel(oracle.gate_grad(z, TAU, g), fd) < 1e-9
    # sigmoid(-z) limits: 1/2 at 0, -> 1 and -> 0 in the tails
    assert abs(oracle.gate_grad(np.array([0.0]), 1.0, np.array([1.0]))[0] - 0.5) < 1e-16
    assert abs(oracle.gate_grad(np.array([-60.0]), 1.0, np.array([1.0]))[0] - 1.0) < 1e-15
    assert oracle.gate_grad(np.array([60.0]), 1.0, np.array([1.0]))[0] < 1e-25


def test_gate_preactivation_gradient_through_the_layer():
    """dL/dz of the layer fed through the gate epilogue equals central finite
    differences in z of the loss computed by the forward recurrence."""
    rng = np.random.default_rng(31)
    T, K, V = 5, 3, 2
    q = rng.standard_normal((T, K))
    k = rng.standard_normal((T, K)) / np.sqrt(K)
    v = rng.standard_normal((T, V))
    z = rng.standard_normal((T, K)) * 2.0 + 3.0
    dO = rng.standard_normal((T, V))
    la = oracle.gate_log_alpha(z, TAU)
    g = oracle.bwd(q, k, v, la, dO, nthreads=1, ckpt=4)
    dz = oracle.gate_grad(z, TAU, g["dlog_alpha"])
    h = 1e-5
    fd = np.zeros_like(z)
    for idx in np.ndindex(z.shape):
        zp = z.copy(); zp[idx] += h
        zm = z.copy(); zm[idx] -= h
        lp = float((oracle.fwd(q, k, v, oracle.gate_log_alpha(zp, TAU), want_state=False, nthreads=1)[0] * dO).sum())
        lm = float((oracle.fwd(q, k, v, oracle.gate_log_alpha(zm, TAU), want_state=False, nthreads=1)[0] * dO).sum())
        fd[idx] = (lp - lm) / (2 * h)
    assert rel(dz, fd) < 1e-7


# ---------------------------------------------------------------- output side

def _og_case(rng, B=2, H=2, T=5, V=6, affine=True):
    o = rng.standard_normal((B, H, T, V)) * 1.5 + 0.3
    g = rng.standard_normal((B, H, T, V)) * 2.0
    w = 1.0 + 0.2 * rng.standard_normal((H, V)) if affine else None
    b = 0.1 * rng.standard_normal((H, V)) if affine else None
    return o, g, w, b


def test_output_gate_closed_forms():
    rng = np.random.default_rng(41)
    o, g, _, _ = _og_case(rng, affine=False)
    # with g -> +inf the gate is the identity (swish(g)/g -> 1): y/g is the
    # normalised row, mean 0 and variance var/(var + eps) per row
    big = np.full_like(g, 40.0)
    y, mu, rstd = oracle.output_gate_fwd(o, big, eps=1e-5)
    xh = y / 40.0
    assert np.abs(xh.mean(-1)).max() < 1e-13
    var = o.var(-1)
    assert np.abs((xh ** 2).mean(-1) - var / (var + 1e-5)).max() < 1e-13
    assert rel(mu, o.mean(-1)) < 1e-15 and rel(rstd, 1.0 / np.sqrt(var + 1e-5)) < 1e-15
    # swish(0) = 0 closes the gate; swish(-inf) -> 0
    assert np.abs(oracle.output_gate_fwd(o, np.zeros_like(g))[0]).max() == 0.0
    assert np.abs(oracle.output_gate_fwd(o, np.full_like(g, -60.0))[0]).max() < 1e-20
    # LN is invariant to a shift and a positive scale of the row
    y1 = oracle.output_gate_fwd(o, g, eps=0.0)[0]
    y2 = oracle.output_gate_fwd(3.0 * o - 7.0, g, eps=0.0)[0]
    assert rel(y2, y1) < 1e-12
    # affine: w = 2, b = 1 gives r (2 xh + 1)
    H, V = o.shape[1], o.shape[3]
    y3 = oracle.output_gate_fwd(o, g, np.full((H, V), 2.0), np.ones((H, V)))[0]
    r = g / (1.0 + np.exp(-g))
    assert rel(y3, 2.0 * oracle.output_gate_fwd(o, g)[0] + r) < 1e-13


@pytest.mark.parametrize("affine", [False, True])
def test_output_gate_gradients_match_central_finite_differences(affine):
    rng = np.random.default_rng(43)
    o, g, w, b = _og_case(rng, B=1, H=2, T=3, V=5, affine=affine)
    dy = rng.standard_normal(o.shape)
    got = oracle.output_gate_bwd(o, g, dy, w, b)
    L = lambda o_, g_, w_, b_: float((oracle.output_gate_fwd(o_, g_, w_, b_)[0] * dy).sum())
    h = 1e-6
    args = {"o": o, "g": g} | ({"w": w, "b": b} if affine else {})
    for name, x in args.items():
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp = x.copy(); xp[idx] += h
            xm = x.copy(); xm[idx] -= h
            ap = dict(args, **{name: xp}); am = dict(args, **{name: xm})
            fd[idx] = (L(ap["o"], ap["g"], ap.get("w"), ap.get("b"))
                       - L(am["o"], am["g"], am.get("w"), am.get("b"))) / (2 * h)
        key = {"o": "do", "g": "dg", "w": "dw", "b": "db"}[name]
        assert rel(got[key], fd) < 1e-7, name


# ---------------------------------------------------------------- scalar gates

def _scalar_case(rng, T=23, K=5, V=4, mu=1.0):
    q = rng.standard_normal((T, K))
    k = rng.standard_normal((T, K)) / np.sqrt(K)
    v = rng.standard_normal((T, V))
    lg = -np.logaddexp(0.0, -(rng.standard_normal(T) + mu))  # log sigmoid, <= 0
    S0 = rng.standard_normal((K, V)) * 0.3
    return q, k, v, lg, S0


def test_scalar_gate_equals_scalar_decay_attention():
    rng = np.random.default_rng(51)
    q, k, v, lg, S0 = _scalar_case(rng)
    o, ST = oracle.scalar_gate_fwd(q, k, v, lg, S0, nthreads=1)
    ro, rST = forms.scalar_decay_attention(q, k, v, lg, S0)
    assert rel(o, ro) < 1e-12 and rel(ST, rST) < 1e-12
    # a constant gamma is RetNet's decay mask
    g = 0.83
    o2, _ = oracle.scalar_gate_fwd(q, k, v, np.full(q.shape[0], np.log(g)), nthreads=1)
    assert rel(o2, forms.decay_mask_attention(q, k, v, g)) < 1e-12
    # batched leading dims are independent heads
    qb = np.stack([q, 2.0 * q]); kb = np.stack([k, k]); vb = np.stack([v, -v]); lb = np.stack([lg, 0.5 * lg])
    ob, _ = oracle.scalar_gate_fwd(qb, kb, vb, lb, nthreads=2)
    assert rel(ob[1], forms.scalar_decay_attention(2.0 * q, k, -v, 0.5 * lg)[0]) < 1e-12


def test_scalar_gate_gradients_match_central_finite_differences():
    """Every gradient of L = sum(o dO) + sum(S_T dS_T) under scalar gates, by
    central differences of the parallel form (which shares nothing with the
    recurrence)."""
    rng = np.random.default_rng(52)
    q, k, v, lg, S0 = _scalar_case(rng, T=7, K=3, V=2)
    dO = rng.standard_normal((7, 2))
    dST = rng.standard_normal((3, 2))
    g = oracle.scalar_gate_bwd(q, k, v, lg, dO, S0=S0, dST=dST, nthreads=1, ckpt=3)
    args = {"q": q, "k": k, "v": v, "log_gamma": lg, "S0": S0}

    def loss(a):
        o, ST = forms.scalar_decay_attention(a["q"], a["k"], a["v"], a["log_gamma"], a["S0"])
        return float((o * dO).sum() + (ST * dST).sum())

    h = 1e-6
    for name, gname in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("log_gamma", "dlog_gamma"), ("S0", "dS0")):
        fd = np.zeros_like(args[name])
        for idx in np.ndindex(args[name].shape):
            ap = {n: x.copy() for n, x in args.items()}; ap[name][idx] += h
            am = {n: x.copy() for n, x in args.items()}; am[name][idx] -= h
            fd[idx] = (loss(ap) - loss(am)) / (2 * h)
        assert g[gname].shape == fd.shape, name
        assert rel(g[gname], fd) < 1e-7, name


# ---------------------------------------------------------------- general gates

def _general_case(rng, T=9, K=4, V=3):
    q = rng.standard_normal((T, K))
    k = rng.standard_normal((T, K)) / np.sqrt(K)
    v = rng.standard_normal((T, V))
    la = -np.logaddexp(0.0, -(rng.standard_normal((T, K)) + 1.0))
    lb = -np.logaddexp(0.0, -(rng.standard_normal((T, V)) + 1.0))
    S0 = rng.standard_normal((K, V)) * 0.3
    return q, k, v, la, lb, S0


def test_general_gate_forward_pins():
    rng = np.random.default_rng(61)
    q, k, v, la, lb, S0 = _general_case(rng)
    o, ST = oracle.general_gate_fwd(q, k, v, la, lb, S0)
    assert rel(o, forms.general_gate_parallel(q, k, v, la, lb, S0)) < 1e-12
    # beta = 1 is the GLA layer of Eq. 3
    o1, S1 = oracle.general_gate_fwd(q, k, v, la, np.zeros_like(v), S0)
    r1, R1 = oracle.fwd(q, k, v, la, S0, nthreads=1)
    assert rel(o1, r1) < 1e-12 and rel(S1, R1) < 1e-12
    # a constant value-side gate gamma on an ungated key side is the decay mask
    o2, _ = oracle.general_gate_fwd(q, k, v, np.zeros_like(q), np.full(v.shape, np.log(0.7)))
    assert rel(o2, forms.decay_mask_attention(q, k, v, 0.7)) < 1e-12
    # leading dims are independent heads
    ob, _ = oracle.general_gate_fwd(np.stack([q, -q]), np.stack([k, k]), np.stack([v, 2 * v]),
                                    np.stack([la, la]), np.stack([lb, 0.5 * lb]))
    assert rel(ob[1], forms.general_gate_parallel(-q, k, 2 * v, la, 0.5 * lb)) < 1e-12


def test_general_gate_gradients_match_central_finite_differences():
    rng = np.random.default_rng(62)
    q, k, v, la, lb, S0 = _general_case(rng, T=5, K=3, V=2)
    dO = rng.standard_normal((5, 2))
    dST = rng.standard_normal((3, 2))
    g = oracle.general_gate_bwd(q, k, v, la, lb, dO, S0, dST)
    args = {"q": q, "k": k, "v": v, "la": la, "lb": lb, "S0": S0}

    def loss(a):
        o, ST = oracle.general_gate_fwd(a["q"], a["k"], a["v"], a["la"], a["lb"], a["S0"])
        return float((o * dO).sum() + (ST * dST).sum())

    h = 1e-6
    for name, gname in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("la", "dlog_alpha"), ("lb", "dlog_beta"),
                        ("S0", "dS0")):
        fd = np.zeros_like(args[name])
        for idx in np.ndindex(args[name].shape):
            ap = {n: x.copy() for n, x in args.items()}; ap[name][idx] += h
            am = {n: x.copy() for n, x in args.items()}; am[name][idx] -= h
            fd[idx] = (loss(ap) - loss(am)) / (2 * h)
        assert rel(g[gname], fd) < 1e-7, name
    # beta = 1 reduces the backward to the GLA one
    g1 = oracle.general_gate_bwd(q, k, v, la, np.zeros_like(v), dO, S0, dST)
    r1 = oracle.bwd(q, k, v, la, dO, S0=S0, dST=dST, nthreads=1, ckpt=2)
    for name in ("dq", "dk", "dv", "dlog_alpha", "dS0"):
        assert rel(g1[name], r1[name]) < 1e-12, name


def test_general_gate_gradients_equal_closed_form():
    """App. C: both gate gradients follow from the other gradients and the
    outputs, without the states."""
    rng = np.random.default_rng(63)
    q, k, v, la, lb, S0 = _general_case(rng, T=17, K=5, V=4)
    dO = rng.standard_normal((17, 4))
    dST = rng.standard_normal((5, 4))
    o, ST = oracle.general_gate_fwd(q, k, v, la, lb, S0)
    g = oracle.general_gate_bwd(q, k, v, la, lb, dO, S0, dST)
    ra, rb = forms.general_gate_closed_form(q, k, v, o, g["dq"], g["dk"], g["dv"], dO, ST, dST)
    assert rel(g["dlog_alpha"], ra) < 1e-12
    assert rel(g["dlog_beta"], rb) < 1e-12
    # state checkpoints every 4 steps instead of 64 recompute the same states
    g4 = oracle.general_gate_bwd(q, k, v, la, lb, dO, S0, dST, ckpt=4)
    for name in g:
        assert np.array_equal(g[name], g4[name]), name


def test_general_gate_closed_form_with_bf16_outputs_has_a_precision_floor():
    """The value-side gate gradient of App. C is a reverse sum over the whole
    sequence of o (.) do - v (.) dv.  With o and dv rounded to bf16 (every
    other value exact) its error at T = 2048 is already 2-3e-2 of its
    magnitude (2.7e-2 here): the floor any bf16 evaluation of that closed
    form over the whole sequence inherits.  Unrounded, the closed form is
    exact (checked above); the state form at chunk boundaries (next test)
    avoids the long sum."""
    import torch
    rng = np.random.default_rng(64)
    T, K, V = 2048, 16, 32
    q = rng.standard_normal((T, K)); k = rng.standard_normal((T, K)) / np.sqrt(K); v = rng.standard_normal((T, V))
    la = -np.logaddexp(0.0, -rng.standard_normal((T, K))) / 16.0
    lb = -np.logaddexp(0.0, -(rng.standard_normal((T, V)) + 2.0))
    dO = rng.standard_normal((T, V))
    o, ST = oracle.general_gate_fwd(q, k, v, la, lb)
    g = oracle.general_gate_bwd(q, k, v, la, lb, dO)
    bf = lambda x: torch.from_numpy(x).float().bfloat16().double().numpy()
    _, rb = forms.general_gate_closed_form(q, k, v, bf(o), g["dq"], g["dk"], bf(g["dv"]), dO)
    err = rel(rb, g["dlog_beta"])
    assert 5e-3 < err < 6e-2, err


def test_value_gate_gradient_carry_is_the_chunk_boundary_state_product():
    """The part of dlog beta beyond a chunk boundary tau is
    colsum(S_tau (.) dS_tau), with dS_tau = dL/dS_tau through the later steps
    (for the last boundary, colsum(S_T (.) dS_T)): the carry the kernels use."""
    rng = np.random.default_rng(65)
    T, K, V, C = 150, 6, 5, 64
    q, k, v, la, lb, S0 = _general_case(rng, T=T, K=K, V=V)
    dO = rng.standard_normal((T, V)); dST = rng.standard_normal((K, V)) * 0.1
    g = oracle.general_gate_bwd(q, k, v, la, lb, dO, S0, dST)
    for tau in (C, 2 * C, T):
        o_a, S_tau = oracle.general_gate_fwd(q[:tau], k[:tau], v[:tau], la[:tau], lb[:tau], S0)
        if tau == T:
            carry = (S_tau * dST).sum(axis=0)
            assert rel(carry, g["dlog_beta"][-1] - (o_a[-1] * dO[-1] - v[-1] * g["dv"][-1])) < 1e-12
        else:
            # dL/dS_tau through the later steps: the backward of the remainder started from S_tau
            rest = oracle.general_gate_bwd(q[tau:], k[tau:], v[tau:], la[tau:], lb[tau:], dO[tau:], S_tau, dST)
            carry = (S_tau * rest["dS0"]).sum(axis=0)
            assert rel(carry, g["dlog_beta"][tau]) < 1e-12
