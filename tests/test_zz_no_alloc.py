"""gla_chunk_fwd_noalloc, the forward that allocates nothing (its workspace is
the library's fixed device scratch array): through the C ABI, its outputs
equal gla_chunk_fwd's bit for bit, on two calls in a row (the second with a
smaller problem, so the array holds the first call's larger contents), and a
problem whose workspace exceeds the array is refused before any launch."""
import ctypes
import sys

import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _inputs(name, io, B, H, T, dk, dv, chunk, subchunk, seed):
    cfg = W._cfg(name, B, H, T, dk, dv, chunk, subchunk, io, seed, gate_mu=0.0, s0_std=0.1)
    inp = W.make_inputs(cfg)
    return cfg, {k: (v.cuda() if v is not None else None) for k, v in inp.items()}


def _via_abi(lib, fn, cfg, d, ws=None):
    import paper_2312_06635_amd as g
    p = g._problem(d["q"], d["v"], cfg["chunk"], cfg["subchunk"], 0, 0.0, d["log_alpha"])
    o = torch.full_like(d["v"], float("nan"))
    ST = torch.full((cfg["B"], cfg["H"], cfg["dk"], cfg["dv"]), float("nan"), device="cuda")
    args = [ctypes.byref(p), g._ptr(d["q"]), g._ptr(d["k"]), g._ptr(d["v"]), g._ptr(d["log_alpha"]),
            g._ptr(d["S0"]), g._ptr(o), g._ptr(ST)]
    if ws is not None:
        args += [g._ptr(ws), ws.numel()]
    st = fn(*args, g._stream(d["q"].device))
    return st, o, ST


def test_noalloc_forward_equals_the_workspace_forward():
    import paper_2312_06635_amd as g
    lib = g.lib()
    cases = [("noalloc_big", "bf16", 2, 3, 700, 256, 512, 64, 16, 71),
             ("noalloc_small", "bf16", 1, 2, 130, 64, 96, 32, 8, 72),
             ("noalloc_f32", "f32", 1, 1, 90, 32, 64, 16, 16, 73)]
    for case in cases:
        cfg, d = _inputs(*case)
        say("case", case)
        need = g.workspace_bytes(cfg["B"], cfg["H"], cfg["T"], cfg["dk"], cfg["dv"], cfg["chunk"], cfg["subchunk"],
                                 d["q"].dtype, op=0)
        assert 0 < need <= g.NOALLOC_SCRATCH_BYTES
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        st1, o1, S1 = _via_abi(lib, lib.gla_chunk_fwd, cfg, d, ws)
        st2, o2, S2 = _via_abi(lib, lib.gla_chunk_fwd_noalloc, cfg, d)
        torch.cuda.synchronize()
        assert st1 == 0 and st2 == 0, (st1, st2)
        assert torch.equal(o1, o2) and torch.equal(S1, S2), case[0]
        # the binding's wrapper reaches the same entry point
        o3, S3 = g.chunk_fwd_noalloc(d["q"], d["k"], d["v"], d["log_alpha"], cfg["chunk"], cfg["subchunk"],
                                     S0=d["S0"], out=(torch.empty_like(o1), torch.empty_like(S1)))
        torch.cuda.synchronize()
        assert torch.equal(o3, o1) and torch.equal(S3, S1), case[0] + " (binding)"
    say("noalloc forward: bit-identical to gla_chunk_fwd")


def test_noalloc_refuses_problems_beyond_the_array():
    import paper_2312_06635_amd as g
    lib = g.lib()
    # a bf16 problem whose forward workspace exceeds the array; no tensor is
    # touched (the refusal comes before any launch), so the pointers are dummies
    B, H, T, dk, dv = 64, 4, 4096, 256, 512
    p = g.GlaProblem(B, H, T, dk, dv, 64, 16, g.GLA_BF16, 0, 0.0)
    assert lib.gla_workspace_bytes(ctypes.byref(p), 0) > g.NOALLOC_SCRATCH_BYTES
    x = torch.zeros(16, device="cuda")
    st = lib.gla_chunk_fwd_noalloc(ctypes.byref(p), x.data_ptr(), x.data_ptr(), x.data_ptr(), None, None,
                                   x.data_ptr(), None, None)
    torch.cuda.synchronize()
    assert st == g.GLA_ERR_SCRATCH
    assert "GLA_ERR_SCRATCH" in lib.gla_status_string(st).decode()
    assert torch.equal(x, torch.zeros(16, device="cuda"))
