"""MI355X-native chunkwise gated linear attention (GLA) layer.

Thin Python binding over the C ABI of ``libgla.so`` (declared in
``include/gla.h``).  This module only marshals arguments: it checks tensors,
allocates outputs and workspace with torch, and passes raw device pointers and
the current HIP stream to the library.  Every step of the computation runs in
the library's HIP kernels; there is no fallback of any kind: every entry point
raises if ``libgla.so`` has not been built.

Layer (paper Sec. 4.1, Eq. 3), per batch row and head:
    S_t = Diag(exp(log_alpha_t)) S_{t-1} + k_t^T v_t,   o_t = q_t S_t.

Example (tensors [B, H, T, d] on the HIP device, bf16 or fp32):
    o, S_T = chunk_fwd(q, k, v, log_alpha, chunk=64, subchunk=16, output_final_state=True)
    g = chunk_bwd(q, k, v, log_alpha, dO, chunk=64, subchunk=16)
    g["dq"], g["dk"], g["dv"], g["dlog_alpha"]
To let the backward reuse the forward's gated operands, size one workspace
with workspace_bytes(..., op=1), pass it to both calls and set
reuse_fwd_workspace=True on the backward.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "chunk_fwd", "chunk_bwd", "recurrent_fwd", "workspace_bytes", "GlaError", "library_path",
    "GLA_OK", "GLA_ERR_NULL", "GLA_ERR_SHAPE", "GLA_ERR_DTYPE", "GLA_ERR_UNSUPPORTED",
    "GLA_ERR_WORKSPACE", "GLA_ERR_HIP", "FLAG_REUSE_FWD_WORKSPACE", "FLAG_SCALAR_GATE", "GlaProblem", "lib",
    "output_gate_fwd", "output_gate_bwd", "output_gate_workspace_bytes", "general_workspace_bytes",
    "SEGMENTS_SHIFT", "FLAG_FP32_DIAGONAL", "chunk_fwd_noalloc", "GLA_ERR_SCRATCH", "NOALLOC_SCRATCH_BYTES",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_HERE, "libgla.so")

GLA_OK, GLA_ERR_NULL, GLA_ERR_SHAPE, GLA_ERR_DTYPE = 0, 1, 2, 3
GLA_ERR_UNSUPPORTED, GLA_ERR_WORKSPACE, GLA_ERR_HIP, GLA_ERR_SCRATCH = 4, 5, 6, 7
NOALLOC_SCRATCH_BYTES = 128 << 20  # GLA_NOALLOC_SCRATCH_BYTES of include/gla.h
GLA_F32, GLA_BF16 = 0, 1
FLAG_REUSE_FWD_WORKSPACE = 1
FLAG_SCALAR_GATE = 2
FLAG_FP32_DIAGONAL = 4
STAGE_SHIFT = 8
SEGMENTS_SHIFT = 16
SEGMENTS_MAX = 0x7FFF


class GlaProblem(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("T", ctypes.c_int32),
                ("dk", ctypes.c_int32), ("dv", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("subchunk", ctypes.c_int32), ("io", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("gate_tau", ctypes.c_float)]


class GlaError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {lib().gla_status_string(status).decode()}")


_lib = None


def lib():
    """The loaded libgla.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(library_path):
            raise ImportError(
                f"{library_path} is missing; build it with `python -m paper_2312_06635_amd.build`")
        L = ctypes.CDLL(library_path)
        P = ctypes.POINTER(GlaProblem)
        vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
        L.gla_workspace_bytes.argtypes = [P, i32]
        L.gla_workspace_bytes.restype = sz
        L.gla_chunk_fwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.gla_chunk_fwd.restype = i32
        L.gla_chunk_fwd_noalloc.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp]
        L.gla_chunk_fwd_noalloc.restype = i32
        L.gla_chunk_bwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.gla_chunk_bwd.restype = i32
        L.gla_recurrent_fwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp]
        L.gla_chunk_fwd_general.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.gla_chunk_fwd_general.restype = i32
        L.gla_recurrent_fwd_general.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.gla_recurrent_fwd_general.restype = i32
        L.gla_chunk_bwd_general.argtypes = [P] + [vp] * 16 + [sz, vp]
        L.gla_chunk_bwd_general.restype = i32
        L.gla_recurrent_fwd.restype = i32
        L.gla_status_string.argtypes = [i32]
        L.gla_status_string.restype = ctypes.c_char_p
        f32 = ctypes.c_float
        L.gla_output_gate_workspace_bytes.argtypes = [P]
        L.gla_output_gate_workspace_bytes.restype = sz
        L.gla_output_gate_fwd.argtypes = [P, vp, vp, vp, vp, f32, vp, vp, vp]
        L.gla_output_gate_fwd.restype = i32
        L.gla_output_gate_bwd.argtypes = [P, vp, vp, vp, vp, f32, vp, vp, vp, vp, vp, vp, sz, vp]
        L.gla_output_gate_bwd.restype = i32
        _lib = L
    return _lib


def _io_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return GLA_BF16
    if dt == torch.float32:
        return GLA_F32
    raise TypeError(f"unsupported dtype {dt}; use torch.bfloat16 or torch.float32")


def _problem(q, v, chunk, subchunk, flags=0, gate_tau=0.0, la=None) -> GlaProblem:
    """la: the gate tensor; a [B, H, T] one selects scalar gates."""
    B, H, T, dk = q.shape
    if la is not None and la.dim() == 3:
        flags |= FLAG_SCALAR_GATE
    return GlaProblem(B, H, T, dk, v.shape[-1], chunk, subchunk, _io_code(q.dtype), flags, float(gate_tau))


def _ptr(t):
    return None if t is None else t.data_ptr()


def _check(q, k, v, la, extra=(), states=()):
    if q.dim() != 4:
        raise ValueError("q must be [B, H, T, d_k]")
    B, H, T, dk = q.shape
    dev = q.device
    if dev.type != "cuda":
        raise ValueError("tensors must be on a HIP device")
    if la is not None and la.dim() == 3:
        # scalar gate: one value per step and head
        if tuple(la.shape) != (B, H, T) or la.device != dev or la.dtype != q.dtype or not la.is_contiguous():
            raise ValueError(f"a scalar log_alpha must be a contiguous {q.dtype} [B, H, T] tensor on {dev}")
        gate = ()
    else:
        gate = (("log_alpha", la, dk),) if la is not None else ()
    for name, t, last in (("k", k, dk),) + gate + (("v", v, None),) + tuple(extra):
        if t.device != dev or t.dtype != q.dtype or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {q.dtype} tensor on {dev}")
        if t.dim() != 4 or t.shape[:3] != (B, H, T) or (last is not None and t.shape[3] != last):
            raise ValueError(f"{name} has shape {tuple(t.shape)}")
    if not q.is_contiguous():
        raise ValueError("q must be contiguous")
    dv = v.shape[3]
    for name, t in states:
        if t is None:
            continue
        if t.device != dev or t.dtype != torch.float32 or not t.is_contiguous() or \
                tuple(t.shape) != (B, H, dk, dv):
            raise ValueError(f"{name} must be a contiguous float32 [B, H, d_k, d_v] tensor on {dev}")


def _stream(dev):
    return torch.cuda.current_stream(dev).cuda_stream


def _segments_flag(segments):
    """GLA_SEGMENTS(n): 0 lets the library decide from the shape."""
    n = int(segments)
    if not 0 <= n <= SEGMENTS_MAX:
        raise ValueError(f"segments must be in [0, {SEGMENTS_MAX}]")
    return n << SEGMENTS_SHIFT


def workspace_bytes(B, H, T, dk, dv, chunk, subchunk, dtype=torch.bfloat16, op=1, scalar_gate=False,
                    segments=0) -> int:
    """Workspace bytes for the forward (op=0) or backward (op=1); scalar_gate
    for a [B, H, T] gate; segments as in chunk_fwd (0 if it does not fit)."""
    flags = (FLAG_SCALAR_GATE if scalar_gate else 0) | _segments_flag(segments)
    p = GlaProblem(B, H, T, dk, dv, chunk, subchunk, _io_code(dtype), flags)
    return int(lib().gla_workspace_bytes(ctypes.byref(p), op))


def general_workspace_bytes(B, H, T, dk, dv, chunk, subchunk, dtype=torch.bfloat16, scalar_gate=False) -> int:
    """Workspace bytes for the general form's backward (op=2); enough for
    every other call on the same problem too."""
    p = GlaProblem(B, H, T, dk, dv, chunk, subchunk, _io_code(dtype), FLAG_SCALAR_GATE if scalar_gate else 0)
    return int(lib().gla_workspace_bytes(ctypes.byref(p), 2))


def _workspace(p, op, dev, workspace):
    need = int(lib().gla_workspace_bytes(ctypes.byref(p), op))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace holds {workspace.numel()} bytes, {need} needed")
    return workspace


def _check_beta(lb, v):
    if lb is None:
        return
    if lb.shape != v.shape or lb.dtype != v.dtype or lb.device != v.device or not lb.is_contiguous():
        raise ValueError(f"log_beta must be a contiguous {v.dtype} tensor shaped like v {tuple(v.shape)}")


def chunk_fwd(q, k, v, log_alpha, chunk=64, subchunk=16, S0=None, output_final_state=False,
              workspace=None, stage=0, out=None, gate_tau=0.0, log_beta=None, segments=0,
              fp32_diagonal=False):
    """Chunkwise GLA forward.  Returns (o, S_T or None).

    log_alpha=None means alpha = 1 (ungated linear attention): no gate tensor
    is read.  A [B, H, T] log_alpha is a scalar gate per step and head (alpha_t =
    gamma_t 1, the scalar-gate rows of Table 1).  gate_tau > 0 means log_alpha holds the gate pre-activation z of
    alpha = sigmoid(z)^(1/gate_tau) (the GLA gate).  stage selects one kernel of the launch sequence (see
    GLA_STAGE_* in include/gla.h); out=(o, S_T) reuses caller-provided output
    tensors.  log_beta ([B, H, T, d_v]) adds the value-side gate of the
    general form G_t = alpha_t^T beta_t (App. C; forward only).  segments
    fixes the sequence segments per head (GLA_SEGMENTS in include/gla.h: 1 =
    states on chip, T/chunk = every chunk's state materialized; 0 = decided
    from the shape).  fp32_diagonal evaluates every diagonal sub-chunk block
    in fp32 log space (GLA_FLAG_FP32_DIAGONAL) instead of on the matrix cores."""
    _check(q, k, v, log_alpha, states=(("S0", S0),))
    _check_beta(log_beta, v)
    B, H, T, dk = q.shape
    dv = v.shape[3]
    flags = (stage << STAGE_SHIFT) | _segments_flag(segments) | (FLAG_FP32_DIAGONAL if fp32_diagonal else 0)
    p = _problem(q, v, chunk, subchunk, flags, gate_tau, log_alpha)
    if out is not None:
        o, ST = out
    else:
        o = torch.empty_like(v)
        ST = torch.empty(B, H, dk, dv, dtype=torch.float32, device=q.device) if output_final_state else None
    ws = _workspace(p, 0, q.device, workspace)
    if log_beta is not None:
        st = lib().gla_chunk_fwd_general(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha),
                                         _ptr(log_beta), _ptr(S0), _ptr(o), _ptr(ST), _ptr(ws),
                                         ws.numel() * ws.element_size(), _stream(q.device))
    else:
        st = lib().gla_chunk_fwd(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(S0),
                                 _ptr(o), _ptr(ST), _ptr(ws), ws.numel() * ws.element_size(),
                                 _stream(q.device))
    if st != GLA_OK:
        raise GlaError(st, "gla_chunk_fwd_general" if log_beta is not None else "gla_chunk_fwd")
    return o, ST


def chunk_fwd_noalloc(q, k, v, log_alpha, chunk=64, subchunk=16, S0=None, out=None, gate_tau=0.0):
    """gla_chunk_fwd_noalloc: the chunkwise forward with the library's fixed
    scratch array as its workspace (nothing is allocated by the library).
    out=(o, S_T or None) must be given (caller-owned outputs); returns it.
    Problems whose forward workspace exceeds NOALLOC_SCRATCH_BYTES raise
    GlaError with status GLA_ERR_SCRATCH."""
    _check(q, k, v, log_alpha, states=(("S0", S0),))
    if out is None:
        raise ValueError("chunk_fwd_noalloc needs out=(o, S_T or None)")
    o, ST = out
    _check(q, k, o, None, states=(("S_T", ST),))
    if o.shape != v.shape:
        raise ValueError("o must be shaped like v")
    p = _problem(q, v, chunk, subchunk, 0, gate_tau, log_alpha)
    st = lib().gla_chunk_fwd_noalloc(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(S0),
                                     _ptr(o), _ptr(ST), _stream(q.device))
    if st != GLA_OK:
        raise GlaError(st, "gla_chunk_fwd_noalloc")
    return o, ST


def chunk_bwd(q, k, v, log_alpha, dO, chunk=64, subchunk=16, S0=None, dST=None,
              want_dS0=False, workspace=None, reuse_fwd_workspace=False, stage=0, out=None,
              gate_tau=0.0, log_beta=None, o=None, segments=0, fp32_diagonal=False):
    """Chunkwise GLA backward for L = sum(o * dO) + sum(S_T * dS_T).

    Returns dict(dq, dk, dv, dlog_alpha, dS0); dlog_alpha is None when
    log_alpha is None (alpha = 1, no gate gradient), shaped like log_alpha
    ([B, H, T] for a scalar gate), and dL/dz when gate_tau > 0
    (log_alpha then holds the gate pre-activation z).  With reuse_fwd_workspace the
    given workspace must still hold what chunk_fwd left for the same inputs.
    stage and out as in chunk_fwd (out is a dict shaped like the result).
    log_beta: the general form's value-side gate (App. C); the result then
    also holds dlog_beta, which needs the forward's output o (without o it is
    None); the workspace must be sized for op=2 (general_workspace_bytes).
    segments and fp32_diagonal as in chunk_fwd (the same segments as the
    forward's when its workspace is reused)."""
    _check(q, k, v, log_alpha, extra=(("dO", dO, v.shape[3]),), states=(("S0", S0), ("dST", dST)))
    _check_beta(log_beta, v)
    _check_beta(o, v)
    B, H, T, dk = q.shape
    dv = v.shape[3]
    flags = (FLAG_REUSE_FWD_WORKSPACE if reuse_fwd_workspace else 0) | (stage << STAGE_SHIFT) | \
        _segments_flag(segments) | (FLAG_FP32_DIAGONAL if fp32_diagonal else 0)
    p = _problem(q, v, chunk, subchunk, flags, gate_tau, log_alpha)
    if reuse_fwd_workspace and workspace is None:
        raise ValueError("reuse_fwd_workspace needs the workspace the forward used")
    if out is not None:
        dq, dkk, dvv, dla, dS0 = (out[n] for n in ("dq", "dk", "dv", "dlog_alpha", "dS0"))
    else:
        dq = torch.empty_like(q)
        dkk = torch.empty_like(k)
        dvv = torch.empty_like(v)
        dla = torch.empty_like(log_alpha) if log_alpha is not None else None
        dS0 = torch.empty(B, H, dk, dv, dtype=torch.float32, device=q.device) if want_dS0 else None
    if log_beta is not None:
        dlb = (out.get("dlog_beta") if out is not None else torch.empty_like(log_beta)) if o is not None else None
        ws = _workspace(p, 2, q.device, workspace)
        st = lib().gla_chunk_bwd_general(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha),
                                         _ptr(log_beta), _ptr(S0), _ptr(o), _ptr(dO), _ptr(dST), _ptr(dq),
                                         _ptr(dkk), _ptr(dvv), _ptr(dla), _ptr(dlb), _ptr(dS0), _ptr(ws),
                                         ws.numel() * ws.element_size(), _stream(q.device))
        if st != GLA_OK:
            raise GlaError(st, "gla_chunk_bwd_general")
        return {"dq": dq, "dk": dkk, "dv": dvv, "dlog_alpha": dla, "dS0": dS0, "dlog_beta": dlb}
    ws = _workspace(p, 1, q.device, workspace)
    st = lib().gla_chunk_bwd(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(S0),
                             _ptr(dO), _ptr(dST), _ptr(dq), _ptr(dkk), _ptr(dvv), _ptr(dla),
                             _ptr(dS0), _ptr(ws), ws.numel() * ws.element_size(),
                             _stream(q.device))
    if st != GLA_OK:
        raise GlaError(st, "gla_chunk_bwd")
    return {"dq": dq, "dk": dkk, "dv": dvv, "dlog_alpha": dla, "dS0": dS0}


def recurrent_fwd(q, k, v, log_alpha, S0=None, output_final_state=False, gate_tau=0.0, log_beta=None):
    """Step-by-step recurrent forward (Eq. 3).  Returns (o, S_T or None);
    log_alpha=None means alpha = 1; log_beta adds the value-side gate of the
    general form (App. C)."""
    _check(q, k, v, log_alpha, states=(("S0", S0),))
    _check_beta(log_beta, v)
    B, H, T, dk = q.shape
    dv = v.shape[3]
    p = _problem(q, v, 16, 16, 0, gate_tau, log_alpha)
    o = torch.empty_like(v)
    ST = torch.empty(B, H, dk, dv, dtype=torch.float32, device=q.device) if output_final_state else None
    if log_beta is not None:
        st = lib().gla_recurrent_fwd_general(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha),
                                             _ptr(log_beta), _ptr(S0), _ptr(o), _ptr(ST), _stream(q.device))
    else:
        st = lib().gla_recurrent_fwd(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha),
                                     _ptr(S0), _ptr(o), _ptr(ST), _stream(q.device))
    if st != GLA_OK:
        raise GlaError(st, "gla_recurrent_fwd")
    return o, ST


def _og_problem(o):
    if o.dim() != 4:
        raise ValueError("o must be [B, H, T, d_v]")
    B, H, T, dv = o.shape
    return GlaProblem(B, H, T, 16, dv, 64, 16, _io_code(o.dtype), 0, 0.0)


def output_gate_workspace_bytes(o):
    """Device workspace (bytes) that output_gate_bwd needs for o's shape when
    the affine gradients are wanted."""
    return int(lib().gla_output_gate_workspace_bytes(ctypes.byref(_og_problem(o))))


def _og_check(o, others, affine):
    if o.device.type != "cuda" or not o.is_contiguous():
        raise ValueError("o must be a contiguous tensor on a HIP device")
    for name, t in others:
        if t.shape != o.shape or t.dtype != o.dtype or t.device != o.device or not t.is_contiguous():
            raise ValueError(f"{name} must match o ({tuple(o.shape)}, {o.dtype})")
    H, dv = o.shape[1], o.shape[3]
    for name, t in affine:
        if t is not None and (tuple(t.shape) != (H, dv) or t.dtype != torch.float32 or t.device != o.device
                              or not t.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous float32 [H, d_v] tensor on {o.device}")


def output_gate_fwd(o, g, ln_w=None, ln_b=None, eps=1e-5, want_stats=False, out=None):
    """Output side of the layer: y = Swish(g) * LN(o) per head row (LN over
    d_v with optional [H, d_v] affine parameters).  Returns (y, stats or None),
    stats = (mean, 1/sqrt(var + eps)) per row, float32 [B, H, T, 2].
    out=(y, stats) reuses preallocated outputs (stats may be None)."""
    _og_check(o, (("g", g),), (("ln_w", ln_w), ("ln_b", ln_b)))
    p = _og_problem(o)
    if out is not None:
        y, stats = out
        _og_check(o, (("y", y),), ())
        if stats is not None and (tuple(stats.shape) != (*o.shape[:3], 2) or stats.dtype != torch.float32
                                  or not stats.is_contiguous()):
            raise ValueError("stats must be a contiguous float32 [B, H, T, 2] tensor")
    else:
        y = torch.empty_like(o)
        stats = torch.empty(*o.shape[:3], 2, dtype=torch.float32, device=o.device) if want_stats else None
    st = lib().gla_output_gate_fwd(ctypes.byref(p), _ptr(o), _ptr(g), _ptr(ln_w), _ptr(ln_b),
                                   ctypes.c_float(eps), _ptr(y), _ptr(stats), _stream(o.device))
    if st != GLA_OK:
        raise GlaError(st, "gla_output_gate_fwd")
    return y, stats


def output_gate_bwd(o, g, dy, ln_w=None, ln_b=None, eps=1e-5, want_affine_grads=True, out=None,
                    workspace=None):
    """Reverse mode of output_gate_fwd for L = sum(y * dy).  Returns dict(do,
    dg, dln_w, dln_b); do is the dO of chunk_bwd; the affine gradients are
    float32 [H, d_v] (None when not wanted).  out=dict(do, dg, dln_w, dln_b)
    reuses preallocated outputs; workspace is a uint8 device tensor of at
    least output_gate_workspace_bytes bytes."""
    _og_check(o, (("g", g), ("dy", dy)), (("ln_w", ln_w), ("ln_b", ln_b)))
    p = _og_problem(o)
    H, dv = o.shape[1], o.shape[3]
    if out is not None:
        d_o, dg, dw, db = out["do"], out["dg"], out.get("dln_w"), out.get("dln_b")
        _og_check(o, (("do", d_o), ("dg", dg)), (("dln_w", dw), ("dln_b", db)))
    else:
        d_o, dg = torch.empty_like(o), torch.empty_like(o)
        dw = torch.empty(H, dv, dtype=torch.float32, device=o.device) if want_affine_grads else None
        db = torch.empty(H, dv, dtype=torch.float32, device=o.device) if want_affine_grads else None
    if workspace is not None:
        ws = workspace
    else:
        need = output_gate_workspace_bytes(o) if (dw is not None or db is not None) else 0
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=o.device)
    st = lib().gla_output_gate_bwd(ctypes.byref(p), _ptr(o), _ptr(g), _ptr(ln_w), _ptr(ln_b),
                                   ctypes.c_float(eps), _ptr(dy), _ptr(d_o), _ptr(dg), _ptr(dw), _ptr(db),
                                   _ptr(ws), ws.numel(), _stream(o.device))
    if st != GLA_OK:
        raise GlaError(st, "gla_output_gate_bwd")
    return {"do": d_o, "dg": dg, "dln_w": dw, "dln_b": db}
