"""Seeded synthetic inputs for the GLA layer workloads.

This module is shared by the tests and the benchmark.  It only draws random
numbers and rounds them to the I/O dtype: it holds none of the layer's
arithmetic, and neither the oracle nor the HIP library imports it.

Recipe (the shapes and gate distribution follow the paper's GLA layers: H=4,
d_k = d/2, d_v = d, gate temperature tau = 16; Sec. 4.4 and Sec. 5.1):
  * one CPU ``torch.Generator`` seeded per workload; draw order
    q, k, v, gate pre-activation x, dO, S0, dS_T;
  * q, k, v, dO ~ N(0, 1) with k scaled by d_k^-1/2;
  * log_alpha = logsigmoid(x) / 16 with x ~ N(mu, 1) (mu = 0, or 2 for the
    slow-decay long-sequence workload);
  * S0, dS_T ~ 0.1 * N(0, 1) in fp32 where a workload asks for them;
  * everything is drawn in fp32 and rounded once (round-to-nearest-even) to
    the I/O dtype; the oracle consumes exactly those rounded values.
No dataset is involved: these tensors stand in for the activations of the
paper's language-model training runs.
"""
from __future__ import annotations

import torch

TAU = 16.0


def _cfg(name, B, H, T, dk, dv, chunk, subchunk, io, seed, gate_mu=0.0, s0_std=0.0,
         want_state=False):
    return dict(name=name, B=B, H=H, T=T, dk=dk, dv=dv, chunk=chunk, subchunk=subchunk, io=io,
                seed=seed, gate_mu=gate_mu, s0_std=s0_std, want_state=want_state)


SWEEP_T = (1024, 2048, 4096, 8192, 16384)

CONFIGS = {
    "tiny_fp32": _cfg("tiny_fp32", 1, 1, 64, 16, 32, 16, 8, "f32", 0),
    "gla1p3b_T2048": _cfg("gla1p3b_T2048", 8, 4, 2048, 256, 512, 64, 16, "bf16", 1),
    "gla340m_T2048": _cfg("gla340m_T2048", 32, 4, 2048, 128, 256, 64, 16, "bf16", 2),
    "long_T16384": _cfg("long_T16384", 1, 4, 16384, 256, 512, 64, 16, "bf16", 3, gate_mu=2.0,
                        s0_std=0.1, want_state=True),
}
for _i, _T in enumerate(SWEEP_T):
    CONFIGS[f"sweep_T{_T}"] = _cfg(f"sweep_T{_T}", 32768 // _T, 16, _T, 128, 128, 64, 16, "bf16",
                                   4 + _i)
# Context only: the shape of the paper's speed comparison of its chunkwise
# kernels (Fig. 2: batch 32, 16 heads of dimension 64, chunk 64, ungated).
CONFIGS["fig2_T2048"] = _cfg("fig2_T2048", 32, 16, 2048, 64, 64, 64, 16, "bf16", 9)


def torch_dtype(io: str) -> torch.dtype:
    return {"f32": torch.float32, "bf16": torch.bfloat16}[io]


def make_inputs(cfg: dict, *, alpha_one: bool = False, dST_std: float = 0.0,
                seed: int | None = None, **overrides) -> dict:
    """Draw one workload's tensors on the CPU.

    Returns q, k, log_alpha [B,H,T,d_k] and v, dO [B,H,T,d_v] in the I/O dtype,
    S0 (or None) and dST (or None) as fp32 [B,H,d_k,d_v].  ``overrides`` may
    replace any shape field (B, H, T, dk, dv) to draw a smaller case with the
    same distributions.  ``alpha_one`` sets log_alpha to 0 after drawing (the
    ungated degenerate case on the same q, k, v).
    """
    c = dict(cfg)
    c.update(overrides)
    B, H, T, dk, dv = c["B"], c["H"], c["T"], c["dk"], c["dv"]
    dt = torch_dtype(c["io"])
    g = torch.Generator().manual_seed(c["seed"] if seed is None else seed)
    q = torch.randn(B, H, T, dk, generator=g)
    k = torch.randn(B, H, T, dk, generator=g) * dk ** -0.5
    v = torch.randn(B, H, T, dv, generator=g)
    x = torch.randn(B, H, T, dk, generator=g) + c["gate_mu"]
    dO = torch.randn(B, H, T, dv, generator=g)
    la = torch.nn.functional.logsigmoid(x) / TAU
    if alpha_one:
        la = torch.zeros_like(la)
    S0 = None
    if c["s0_std"] > 0:
        S0 = torch.randn(B, H, dk, dv, generator=g) * c["s0_std"]
    dST = None
    if dST_std > 0:
        dST = torch.randn(B, H, dk, dv, generator=g) * dST_std
    out = dict(q=q.to(dt), k=k.to(dt), v=v.to(dt), log_alpha=la.to(dt), dO=dO.to(dt), S0=S0,
               dST=dST)
    return out

