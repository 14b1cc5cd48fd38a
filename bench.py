#!/usr/bin/env python3
"""Benchmark of the chunkwise GLA layer, forward + backward, on one MI355X.

One step = the whole hot path over one batch: gla_chunk_fwd (gate factors,
gated operands and intra-chunk matrices; state pass and outputs) followed by
gla_chunk_bwd reusing the forward's workspace (dq sweep; dk/dlog_alpha sweep;
dv sweep).  Each stage is launched on its own through the C ABI's stage
selector with a HIP event after it, so the per-kernel durations are measured
live on the stream the kernels run on, inside the timed region.  With
--output-gate the step also runs the output side (per-head LayerNorm and Swish
output gate, Sec. 4.4) after the forward and its reverse mode, which produces
the dO the backward sweeps consume, before them.

Prints one JSON line.  `value` is tokens/s (B*T per step) with all inputs
resident in HBM; TFLOP/s uses the algorithmic FLOP count of the chunk form
(per token-head: fwd 4 d_k d_v + (C+1)(d_k+d_v), bwd 8 d_k d_v + (C+1)(3 d_k + 2 d_v)).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import torch  # noqa: E402

import workloads as W  # noqa: E402

PEAK_BF16_FLOPS = 2.5e15
PEAK_F32_FLOPS = 157.3e12
PEAK_HBM = 8.0e12
RIDGE = PEAK_BF16_FLOPS / PEAK_HBM

STAGES = [("prep", "fwd", 1), ("fwd_main", "fwd", 2), ("bwd_dq", "bwd", 2), ("bwd_intra", "bwd", 3),
          ("bwd_dk", "bwd", 4), ("bwd_dv", "bwd", 5)]
# with the output side (Sec. 4.4): LN + Swish gate after the forward, its
# reverse mode (producing the layer's dO) before the backward sweeps
STAGES_OG = STAGES[:2] + [("og_fwd", "og", 0), ("og_bwd", "og", 1)] + STAGES[2:]
# the general form (App. C, value-side gate beta): its backward's stages
STAGES_GB = STAGES[:2] + [("beta_prep", "bwdg", 2), ("bwd_dq", "bwdg", 3), ("bwd_intra", "bwdg", 4),
                          ("bwd_dk", "bwdg", 5), ("bwd_dv", "bwdg", 6), ("beta_grad", "bwdg", 7)]


def algorithmic(cfg, gate=True, scalar_gate=False, value_gate=False):
    """Algorithmic FLOPs and HBM bytes per launch of each stage (and totals).

    "bytes" counts only the layer's own I/O that the kernel reads or writes
    (q, k, log alpha, v, dO in; o, dq, dk, dv, dlog alpha out; s bytes per
    element), the per-kernel share of the s (9 d_k + 5 d_v) per token-head of
    the whole layer; "bytes_all" adds the intermediates the kernel moves
    through the workspace (gated operands, P, the backward's hand-offs), which
    the measured traffic is compared against.  FLOPs split the chunk form's
    algorithmic count over the kernels (fwd 4 d_k d_v + (C+1)(d_k + d_v), bwd
    8 d_k d_v + (C+1)(3 d_k + 2 d_v) per token-head).  gate=False is the
    alpha = 1 layer (no gate read, no gate gradient); scalar_gate has one gate
    value per step and head."""
    B, H, T, K, V, C = cfg["B"], cfg["H"], cfg["T"], cfg["dk"], cfg["dv"], cfg["chunk"]
    ga = (1.0 / K if scalar_gate else 1.0) if gate else 0.0  # gate elements per step, in units of K
    s = 2 if cfg["io"] == "bf16" else 4
    n = B * H * T                       # token-heads
    N = (T + C - 1) // C
    g = B * H * N * K * 4               # chunk decays (fp32)
    P = n * C * s                       # intra-chunk matrices
    qk = n * s * K                      # one [B, H, T, d_k] io tensor
    vv = n * s * V                      # one [B, H, T, d_v] io tensor
    la = qk * ga                        # the gate tensor (or its gradient)
    st = {
        # gate factors, Q (.) Lambda, K (.) Gamma, P: reads q, k, log alpha
        "prep": dict(flops=n * (C + 1) * K, bytes=2 * qk + la, inter=2 * qk + P + g),
        # state pass + output: reads v (and log beta); writes o
        "fwd_main": dict(flops=n * (4 * K * V + (C + 1) * V), bytes=(3 if value_gate else 2) * vv,
                         inter=2 * qk + P + g),
        # dq sweep (and dP): reads k, log alpha, v, dO
        "bwd_dq": dict(flops=n * (2 * K * V + (C + 1) * V), bytes=qk + la + 2 * vv, inter=n * K * 4 + n * C * 4),
        # intra-chunk terms: reads q, k, log alpha; writes dq
        "bwd_intra": dict(flops=n * (C + 1) * 3 * K, bytes=2 * qk + la + qk,
                          inter=n * C * 4 + n * K * 4 + 2 * qk + B * H * N * K * 4),
        # dk sweep: reads q, k, log alpha, v, dO; writes dk, dlog alpha
        "bwd_dk": dict(flops=n * 4 * K * V, bytes=2 * qk + la + 2 * vv + qk + la,
                       inter=2 * qk + n * K * 4 + B * H * N * K * 4),
        # dv sweep: reads dO; writes dv
        "bwd_dv": dict(flops=n * (2 * K * V + (C + 1) * V), bytes=2 * vv, inter=2 * qk + P + g),
        # output side: reads o, g and the [H, d_v] affine; writes y
        "og_fwd": dict(flops=n * V * 12, bytes=3 * vv + H * V * 8, inter=0),
        # its reverse: reads o, g, dy and the affine; writes dO, dg, dw, db
        "og_bwd": dict(flops=n * V * 24, bytes=5 * vv + H * V * 16, inter=0),
        # general form: Vh, Oh from v, dO, log beta
        "beta_prep": dict(flops=n * V * 6, bytes=3 * vv, inter=2 * vv),
        # dlog beta: reads o, dO, v, dv; writes dlog beta
        "beta_grad": dict(flops=n * V * 4, bytes=5 * vv, inter=0),
    }
    if value_gate:  # the dv sweep also reads log beta
        st["bwd_dv"]["bytes"] += vv
    for a in st.values():
        a["bytes_all"] = a["bytes"] + a.pop("inter")
    fwd = n * (4 * K * V + (C + 1) * (K + V))
    bwd = n * (8 * K * V + (C + 1) * (3 * K + 2 * V))
    io_bytes = n * s * ((7 + 2 * ga) * K + 5 * V)
    return st, fwd, bwd, io_bytes


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def tiny_single_thread_ms(reps=20):
    """The oracle's forward + backward on the tiny fp32 workload (B=1, H=1,
    T=64, d_k=16, d_v=32) with one thread: median wall time of reps runs."""
    import oracle
    cfg = W.CONFIGS["tiny_fp32"]
    inp = W.make_inputs(cfg)
    f = lambda t: None if t is None else t.float().reshape(-1, *t.shape[2:]).double().numpy()
    q, k, v, la, dO = (f(inp[n]) for n in ("q", "k", "v", "log_alpha", "dO"))
    times = []
    for _ in range(reps):
        t0 = time.perf_counter()
        oracle.fwd(q, k, v, la, nthreads=1)
        oracle.bwd(q, k, v, la, dO, nthreads=1)
        times.append(time.perf_counter() - t0)
    times.sort()
    return 1e3 * times[len(times) // 2]


def cpu_baseline(cfg, inputs, target_s=15.0):
    """The fp64 oracle timed on the host cores on a bounded sample of heads."""
    import numpy as np

    import oracle

    oracle.build()
    threads = oracle.default_threads()
    BH = cfg["B"] * cfg["H"]
    flat = {k: (v.float().reshape(BH, *v.shape[2:]) if v is not None else None) for k, v in inputs.items()}
    # calibrate on one head, then size the sample to ~target_s of wall time
    def run(idx, nth):
        sl = lambda n: None if flat[n] is None else flat[n][idx].double().numpy()
        t0 = time.perf_counter()
        oracle.fwd(sl("q"), sl("k"), sl("v"), sl("log_alpha"), sl("S0"), nthreads=nth)
        oracle.bwd(sl("q"), sl("k"), sl("v"), sl("log_alpha"), sl("dO"), S0=sl("S0"), dST=sl("dST"),
                   nthreads=nth)
        return time.perf_counter() - t0
    t1 = run([0], 1)
    heads = int(max(1, min(BH, threads * max(1, int(target_s / max(t1, 1e-3))))))
    heads = max(1, min(BH, (heads // threads) * threads if heads >= threads else heads))
    idx = list(range(heads))
    el, reps = 0.0, 0
    while reps == 0 or el < 0.6 * target_s:  # whole passes over the sample until ~target_s of wall time
        el += run(idx, threads)
        reps += 1
    tokens = reps * heads * cfg["T"] / cfg["H"]
    del np
    return {"value": tokens / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{heads} of {BH} heads (full T={cfg['T']}) x {reps} passes, fwd+bwd fp64 recurrence + "
                      f"BPTT, {el:.1f} s wall; tokens counted as heads*T/H per pass",
            "cpu_model": cpu_model(),
            # one thread, this workload: one head's fwd+bwd measured (the
            # calibration run above), the whole step as BH independent heads
            "single_thread_one_head_s": round(t1, 3),
            "single_thread_step_s": round(t1 * BH, 1),
            "tiny_fp32_single_thread_ms": round(tiny_single_thread_ms(), 4)}


COPY_BYTES = 1 << 30


def calibrate_copy():
    """A plain streaming kernel that reads and writes COPY_BYTES once each (an
    element-wise multiply by one): the reference whose FETCH_SIZE / WRITE_SIZE
    counters scale those of the layer's kernels."""
    dev = torch.device("cuda:0")
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "launches": 3}), flush=True)


def source_digest():
    """Hash of the kernel sources, to tell whether stored counters are current."""
    import hashlib
    h = hashlib.sha256()
    cdir = os.path.join(ROOT, "paper_2312_06635_amd", "csrc")
    for name in sorted(os.listdir(cdir)):
        with open(os.path.join(cdir, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary, or
    None when there is none or the kernels changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    digest, found = None, None
    with open(path) as f:
        for line in f:
            line = line.strip()
            if line.startswith("source_digest:"):
                digest = line.split(":", 1)[1].strip()
            if line.startswith(f"traffic_bytes[{kernel}]:"):
                found = float(line.split(":", 1)[1].strip())
    if digest != source_digest():
        return None
    return found


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="gla1p3b_T2048", choices=sorted(W.CONFIGS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gate", action="store_true",
                    help="the alpha = 1 (ungated) layer: log_alpha passed as NULL")
    ap.add_argument("--gate-tau", type=float, default=0.0,
                    help="> 0: pass the gate pre-activation z (alpha = sigmoid(z)^(1/tau)) instead of log alpha")
    ap.add_argument("--scalar-gate", action="store_true",
                    help="one gate value per step and head (log gamma [B, H, T], Table 1's scalar gates)")
    ap.add_argument("--value-gate", action="store_true",
                    help="general form G = alpha^T beta (App. C): adds log beta [B, H, T, d_v]")
    ap.add_argument("--output-gate", action="store_true",
                    help="include the output side (per-head LN + Swish gate, Sec. 4.4) in the step")
    ap.add_argument("--segments", type=int, default=0,
                    help="fix the sequence segments per head (GLA_SEGMENTS: 1 = states on chip, T/chunk = every "
                         "chunk's state materialized in HBM); 0 = the library's choice")
    ap.add_argument("--fp32-diagonal", action="store_true",
                    help="every diagonal sub-chunk block in fp32 log space (GLA_FLAG_FP32_DIAGONAL)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy (reference for HBM traffic counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: heads shard across GPUs with no communication, "
              "and no multi-GPU path is built.", file=sys.stderr)
        sys.exit(2)

    if args.calibrate_copy:
        calibrate_copy()
        return

    import paper_2312_06635_amd as gla

    cfg = W.CONFIGS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    inp_cpu = W.make_inputs(cfg, alpha_one=args.no_gate)
    d = {k: (v.to(dev) if v is not None else None) for k, v in inp_cpu.items()}
    if args.scalar_gate:
        # log gamma = logsigmoid(x) / 16 per (batch row, head, step), the
        # per-feature recipe with one draw per step
        gs = torch.Generator().manual_seed(cfg["seed"] + 5)
        lg = torch.nn.functional.logsigmoid(torch.randn(cfg["B"], cfg["H"], cfg["T"], generator=gs)) / 16.0
        inp_cpu["log_alpha"] = lg.to(inp_cpu["q"].dtype)
        d["log_alpha"] = inp_cpu["log_alpha"].to(dev)
    if args.no_gate:
        d["log_alpha"] = None
    elif args.gate_tau > 0:
        # gate pre-activations; log alpha = logsigmoid(z) / tau is formed in the kernels
        gz = torch.Generator().manual_seed(cfg["seed"] + 7)
        z = torch.randn(inp_cpu["log_alpha"].shape, generator=gz) * 2.0 + 1.0  # [B, H, T] with --scalar-gate
        d["log_alpha"] = z.to(dtype=d["q"].dtype, device=dev)
        inp_cpu["log_alpha"] = torch.nn.functional.logsigmoid(z.double()).div(args.gate_tau).to(inp_cpu["q"].dtype)
    B, H, T, K, V, C, c = (cfg[x] for x in ("B", "H", "T", "dk", "dv", "chunk", "subchunk"))
    dt = d["q"].dtype
    ws = torch.empty(gla.workspace_bytes(B, H, T, K, V, C, c, dt, op=1, scalar_gate=args.scalar_gate,
                                         segments=args.segments), dtype=torch.uint8, device=dev)
    if ws.numel() == 0:
        print(f"--segments {args.segments} does not fit this workload (it must divide T/chunk = {T // C})",
              file=sys.stderr)
        sys.exit(2)
    o = torch.empty_like(d["v"])
    ST = torch.empty(B, H, K, V, dtype=torch.float32, device=dev) if cfg["want_state"] else None
    grads = {"dq": torch.empty_like(d["q"]), "dk": torch.empty_like(d["k"]), "dv": torch.empty_like(d["v"]),
             "dlog_alpha": torch.empty_like(d["log_alpha"]) if d["log_alpha"] is not None else None,
             "dS0": torch.empty(B, H, K, V, dtype=torch.float32, device=dev) if d["S0"] is not None else None}
    stream = torch.cuda.current_stream(dev)
    stages = STAGES_OG if args.output_gate else STAGES
    if args.value_gate:
        if args.output_gate or args.gate_tau > 0 or args.segments > 1:
            print("--value-gate does not combine with --output-gate, --gate-tau or --segments", file=sys.stderr)
            sys.exit(2)
        stages = STAGES_GB
        gb = torch.Generator().manual_seed(cfg["seed"] + 13)
        # log beta = logsigmoid(x) / 16, x ~ N(0, 1), the key gate's recipe on the value side
        d["log_beta"] = (torch.nn.functional.logsigmoid(torch.randn(B, H, T, V, generator=gb)) / 16.0).to(dt).to(dev)
        ws = torch.empty(gla.general_workspace_bytes(B, H, T, K, V, C, c, dt, scalar_gate=args.scalar_gate),
                         dtype=torch.uint8, device=dev)
        grads["dlog_beta"] = torch.empty_like(d["v"])
    if args.output_gate:
        # output-gate pre-activations, the loss gradient at y and the LN affine
        go = torch.Generator().manual_seed(cfg["seed"] + 11)
        og = {"g": torch.randn(B, H, T, V, generator=go).to(dt), "dy": torch.randn(B, H, T, V, generator=go).to(dt),
              "w": 1.0 + 0.1 * torch.randn(H, V, generator=go), "b": 0.1 * torch.randn(H, V, generator=go)}
        og = {k: v.to(dev) for k, v in og.items()}
        y = torch.empty_like(o)
        og_out = {"do": torch.empty_like(o), "dg": torch.empty_like(o),
                  "dln_w": torch.empty(H, V, dtype=torch.float32, device=dev),
                  "dln_b": torch.empty(H, V, dtype=torch.float32, device=dev)}
        og_ws = torch.empty(max(gla.output_gate_workspace_bytes(o), 1), dtype=torch.uint8, device=dev)
        d["dO"] = og_out["do"]  # the layer's dO is what the output side's reverse mode produces

    def launch(stage_name, which, stage):
        if which == "og":
            if stage == 0:
                gla.output_gate_fwd(o, og["g"], og["w"], og["b"], out=(y, None))
            else:
                gla.output_gate_bwd(o, og["g"], og["dy"], og["w"], og["b"], out=og_out, workspace=og_ws)
        elif which == "bwdg":
            gla.chunk_bwd(d["q"], d["k"], d["v"], d["log_alpha"], d["dO"], C, c, S0=d["S0"], dST=d["dST"],
                          workspace=ws, reuse_fwd_workspace=True, stage=stage, out=grads,
                          log_beta=d["log_beta"], o=o, fp32_diagonal=args.fp32_diagonal)
        elif which == "fwd":
            gla.chunk_fwd(d["q"], d["k"], d["v"], d["log_alpha"], C, c, S0=d["S0"], workspace=ws,
                          stage=stage, out=(o, ST), gate_tau=args.gate_tau, log_beta=d.get("log_beta"),
                          segments=args.segments, fp32_diagonal=args.fp32_diagonal)
        else:
            gla.chunk_bwd(d["q"], d["k"], d["v"], d["log_alpha"], d["dO"], C, c, S0=d["S0"], dST=d["dST"],
                          workspace=ws, reuse_fwd_workspace=True, stage=stage, out=grads,
                          gate_tau=args.gate_tau, segments=args.segments, fp32_diagonal=args.fp32_diagonal)

    def step(events=None):
        if events is not None:
            events[0].record(stream)
        for i, (nm, which, stg) in enumerate(stages):
            launch(nm, which, stg)
            if events is not None:
                events[i + 1].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    stage_ms = {nm: 0.0 for nm, _, _ in stages}
    for s in range(args.steps):
        for i, (nm, _, _) in enumerate(stages):
            stage_ms[nm] += evs[s][i].elapsed_time(evs[s][i + 1]) / args.steps
    st_alg, fwd_flops, bwd_flops, io_bytes = algorithmic(cfg, gate=not args.no_gate, scalar_gate=args.scalar_gate,
                                                         value_gate=args.value_gate)
    if args.value_gate:
        io_bytes += 3 * B * H * T * V * (2 if cfg["io"] == "bf16" else 4)  # log beta in, o into the backward, dlog beta out
    if args.output_gate:
        io_bytes += st_alg["og_fwd"]["bytes"] + st_alg["og_bwd"]["bytes"]
    ms_per_step = 1e3 * elapsed / args.steps
    tokens = B * T
    value = tokens * args.steps / elapsed
    tflops = (fwd_flops + bwd_flops) * args.steps / elapsed / 1e12
    peak = PEAK_BF16_FLOPS if cfg["io"] == "bf16" else PEAK_F32_FLOPS

    def roofline(nm):
        a, t = st_alg[nm], stage_ms[nm] * 1e-3
        if a["flops"] / a["bytes"] < RIDGE:
            r = {"kernel": nm, "bound": "hbm", "achieved": a["bytes"] / t / 1e9, "peak": PEAK_HBM / 1e9,
                 "unit": "GB/s"}
        else:
            r = {"kernel": nm, "bound": "mfma", "achieved": a["flops"] / t / 1e12, "peak": peak / 1e12,
                 "unit": "TFLOP/s"}
        r["frac"] = r["achieved"] / r["peak"]
        return r

    dom = max(stage_ms, key=stage_ms.get)
    roof = roofline(dom)
    plain = not (args.no_gate or args.gate_tau > 0 or args.output_gate or args.scalar_gate or args.value_gate or
                 args.segments or args.fp32_diagonal)
    roof["traffic"] = measured_traffic(args.workload, dom) if plain else None
    roof["avg_ms"] = stage_ms[dom]
    # the kernel's own share of the layer I/O (what "achieved" divides) and the
    # bytes it moves including workspace intermediates; measured traffic is
    # compared with the former
    roof["algorithmic_bytes"] = st_alg[dom]["bytes"]
    roof["bytes_with_intermediates"] = st_alg[dom]["bytes_all"]
    roof["traffic_ratio"] = (roof["traffic"] / st_alg[dom]["bytes"]) if roof["traffic"] else None
    stage_frac = {nm: f"{r['frac']:.3f} of {r['bound']}" for nm, r in ((nm, roofline(nm)) for nm in stage_ms)}

    out = {
        "metric": "GLA fwd+bwd tokens/s and TFLOP/s (% bf16 MFMA peak), 1.3B layer, T=2048",
        "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg["io"], "data": "synthetic",
        "config": {"workload": args.workload, "B": B, "H": H, "T": T, "d_k": K, "d_v": V, "chunk": C,
                   "subchunk": c, "parallelism": "none (1 GPU)",
                   **({"gate": "none (alpha = 1, log_alpha NULL)"} if args.no_gate else {}),
                   **({"gate": f"pre-activation z, alpha = sigmoid(z)^(1/{args.gate_tau:g})"}
                      if args.gate_tau > 0 else {}),
                   **({"gate_shape": "scalar per step and head, log gamma [B, H, T]"} if args.scalar_gate else {}),
                   **({"value_gate": "general form alpha^T beta, log beta [B, H, T, d_v]"}
                      if args.value_gate else {}),
                   **({"output_side": "per-head LN (affine) + Swish output gate, fwd + bwd"}
                      if args.output_gate else {}),
                   **({"segments": args.segments} if args.segments else {}),
                   **({"diagonal_blocks": "fp32 log space"} if args.fp32_diagonal else {})},
        "tflops": tflops, "mfma_peak_frac": tflops * 1e12 / peak,
        "hbm_io_roofline_frac": (io_bytes / PEAK_HBM) / (elapsed / args.steps),
        "stage_ms": {k: round(v, 4) for k, v in stage_ms.items()},
        "stage_roofline_frac": stage_frac,
        "roofline": roof,
    }
    if not args.no_cpu_baseline and not args.scalar_gate and not args.value_gate:
        out["cpu_baseline"] = cpu_baseline(cfg, inp_cpu)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
