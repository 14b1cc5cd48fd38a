"""The Python binding on the CPU: it refuses tensors that are not on a HIP
device, malformed shapes and out-of-range options before reaching the
library, fails loudly when libgla.so is missing (there is no fallback), and
its size helpers agree with the C ABI.  No call here launches a kernel."""
import ctypes

import pytest
import torch

import paper_2312_06635_amd as gla
from paper_2312_06635_amd import build as glabuild


@pytest.fixture(scope="module", autouse=True)
def built():
    import os
    if not os.path.exists(gla.library_path):
        glabuild.build()


def cpu_inputs(B=1, H=2, T=64, dk=32, dv=48, dtype=torch.bfloat16):
    g = torch.Generator().manual_seed(0)
    q, k = (torch.randn(B, H, T, dk, generator=g).to(dtype) for _ in range(2))
    v, dO = (torch.randn(B, H, T, dv, generator=g).to(dtype) for _ in range(2))
    la = (-torch.rand(B, H, T, dk, generator=g)).to(dtype)
    return q, k, v, la, dO


def test_host_tensors_are_refused():
    q, k, v, la, dO = cpu_inputs()
    with pytest.raises(ValueError, match="HIP device"):
        gla.chunk_fwd(q, k, v, la)
    with pytest.raises(ValueError, match="HIP device"):
        gla.chunk_bwd(q, k, v, la, dO)
    with pytest.raises(ValueError, match="HIP device"):
        gla.recurrent_fwd(q, k, v, la)


def test_malformed_shapes_are_refused():
    q, k, v, la, dO = cpu_inputs()
    with pytest.raises(ValueError, match=r"\[B, H, T, d_k\]"):
        gla.chunk_fwd(q[0], k, v, la)


def test_segment_option_range():
    assert gla._segments_flag(0) == 0
    assert gla._segments_flag(8) == 8 << gla.SEGMENTS_SHIFT
    for bad in (-1, gla.SEGMENTS_MAX + 1):
        with pytest.raises(ValueError):
            gla._segments_flag(bad)


def test_workspace_helpers_match_the_c_abi():
    L = gla.lib()
    for kw in (dict(B=2, H=3, T=200, dk=64, dv=128), dict(B=1, H=4, T=16384, dk=256, dv=512)):
        for op in (0, 1):
            p = gla.GlaProblem(kw["B"], kw["H"], kw["T"], kw["dk"], kw["dv"], 64, 16, gla.GLA_BF16, 0, 0.0)
            assert gla.workspace_bytes(**kw, chunk=64, subchunk=16, op=op) == L.gla_workspace_bytes(ctypes.byref(p), op)
    # a segment count that does not divide T / C has no workspace (the calls refuse it)
    assert gla.workspace_bytes(1, 1, 256, 64, 64, 64, 16, segments=3) == 0
    assert gla.workspace_bytes(1, 1, 256, 64, 64, 64, 16, segments=4) > gla.workspace_bytes(1, 1, 256, 64, 64, 64, 16,
                                                                                           segments=1)
    assert gla.general_workspace_bytes(2, 3, 200, 64, 128, 64, 16) > gla.workspace_bytes(2, 3, 200, 64, 128, 64, 16)


def test_scalar_gate_is_selected_by_the_gate_shape():
    q, k, v, la, dO = cpu_inputs()
    assert gla._problem(q, v, 64, 16, 0, 0.0, la).flags & gla.FLAG_SCALAR_GATE == 0
    assert gla._problem(q, v, 64, 16, 0, 0.0, la[..., 0]).flags & gla.FLAG_SCALAR_GATE


def test_errors_carry_the_library_status_string():
    e = gla.GlaError(gla.GLA_ERR_WORKSPACE, "gla_chunk_fwd")
    assert e.status == gla.GLA_ERR_WORKSPACE and "GLA_ERR_WORKSPACE" in str(e)


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(gla, "_lib", None)
    monkeypatch.setattr(gla, "library_path", str(tmp_path / "libgla.so"))
    with pytest.raises(ImportError, match="missing"):
        gla.lib()
    with pytest.raises(ImportError):
        gla.workspace_bytes(1, 1, 64, 16, 32, 16, 8)
