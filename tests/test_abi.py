"""The C-ABI library: it loads, exports every symbol include/gla.h declares (and
nothing else), and rejects bad arguments before touching the device.  CPU only:
no call here reaches a kernel launch."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2312_06635_amd as gla
from paper_2312_06635_amd import build as glabuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gla.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(gla.library_path):
        glabuild.build()
    return gla.lib()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(gla_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    assert declared_functions() == ["gla_chunk_bwd", "gla_chunk_bwd_general", "gla_chunk_fwd", "gla_chunk_fwd_general",
                                    "gla_chunk_fwd_noalloc",
                                    "gla_output_gate_bwd", "gla_output_gate_fwd",
                                    "gla_output_gate_workspace_bytes", "gla_recurrent_fwd",
                                    "gla_recurrent_fwd_general", "gla_status_string", "gla_workspace_bytes"]


def test_header_is_plain_c(tmp_path):
    """include/gla.h compiles as strict C99 and C++17 (no warnings), with every
    flag and macro usable from C."""
    src = tmp_path / "use.c"
    src.write_text(
        '#include "gla.h"\n'
        "int main(void) {\n"
        "  gla_problem p = {1, 1, 64, 16, 32, 16, 8, GLA_BF16, 0, 0.0f};\n"
        "  p.flags = GLA_FLAG_REUSE_FWD_WORKSPACE | GLA_FLAG_SCALAR_GATE | GLA_FLAG_FP32_DIAGONAL |\n"
        "            (2u << GLA_STAGE_SHIFT) | GLA_SEGMENTS(4);\n"
        "  return (p.flags & (unsigned)GLA_SEGMENTS_MASK) == GLA_SEGMENTS(4) &&\n"
        "         (p.flags & (unsigned)GLA_STAGE_MASK) >> GLA_STAGE_SHIFT == 2u ? 0 : 1;\n"
        "}\n")
    inc = os.path.join(ROOT, "include")
    for cmd in (["gcc", "-std=c99"], ["g++", "-std=c++17", "-x", "c++"]):
        exe = tmp_path / cmd[0]
        subprocess.run(cmd + ["-Wall", "-Wextra", "-pedantic", "-Werror", "-I", inc, str(src), "-o", str(exe)],
                       check=True, capture_output=True, text=True)
        assert subprocess.run([str(exe)]).returncode == 0


def test_every_declared_symbol_is_exported(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def test_only_the_boundary_is_exported(L):
    out = subprocess.run(["nm", "-D", "--defined-only", gla.library_path], capture_output=True,
                         text=True, check=True).stdout
    syms = {line.split()[-1] for line in out.splitlines() if " T " in line}
    assert set(declared_functions()) <= syms
    assert not [s for s in syms if s.startswith("gla_") and s not in declared_functions()]


def test_status_strings(L):
    for code in range(8):
        s = L.gla_status_string(code).decode()
        assert s.startswith("GLA_OK" if code == 0 else "GLA_ERR")
    assert L.gla_status_string(99).decode() == "GLA_ERR_UNKNOWN"


def P(**kw):
    base = dict(B=2, H=3, T=200, dk=64, dv=128, chunk=64, subchunk=16, io=gla.GLA_BF16, flags=0)
    base.update(kw)
    return gla.GlaProblem(**base)


def test_workspace_bytes(L):
    p = P()
    fwd = L.gla_workspace_bytes(ctypes.byref(p), 0)
    bwd = L.gla_workspace_bytes(ctypes.byref(p), 1)
    BH, T, K, C, N = 6, 200, 64, 64, 4
    assert fwd >= 2 * BH * T * K * 2 + BH * N * C * C * 2 + BH * N * K * 4
    assert bwd >= fwd + BH * N * C * C * 4
    assert fwd % 256 == 0 and bwd % 256 == 0
    p32 = P(io=gla.GLA_F32)
    assert L.gla_workspace_bytes(ctypes.byref(p32), 0) > fwd
    assert L.gla_workspace_bytes(ctypes.byref(p), 2) > bwd  # the general form's backward
    assert L.gla_workspace_bytes(ctypes.byref(p), -1) == 0
    assert L.gla_workspace_bytes(None, 0) == 0
    assert L.gla_workspace_bytes(ctypes.byref(P(dk=24)), 0) == 0


def test_scalar_gate_workspace(L):
    """A scalar gate adds the per-key-tile gate-gradient sums to the backward's
    workspace (B H ceil(d_k/32) T fp32) and nothing to the forward's."""
    for dk, T in ((64, 200), (48, 77), (256, 2048)):
        p, ps = P(dk=dk, T=T), P(dk=dk, T=T, flags=gla.FLAG_SCALAR_GATE)
        assert L.gla_workspace_bytes(ctypes.byref(ps), 0) == L.gla_workspace_bytes(ctypes.byref(p), 0)
        extra = L.gla_workspace_bytes(ctypes.byref(ps), 1) - L.gla_workspace_bytes(ctypes.byref(p), 1)
        need = 6 * ((dk + 31) // 32) * T * 4
        assert need <= extra < need + 256


def test_sequence_segments_workspace(L):
    """Few heads and a long sequence: the workspace holds the segments'
    initial and local final states (forward) and final-state gradients
    (backward) -- 8 segments for 4 heads of 16384 steps at d_k 256, d_v 512 --
    and none when the sequence does not divide into whole chunks."""
    p = P(B=1, H=4, T=16384, dk=256, dv=512)
    f, b = L.gla_workspace_bytes(ctypes.byref(p), 0), L.gla_workspace_bytes(ctypes.byref(p), 1)
    states = 4 * 8 * 256 * 512 * 4
    kernels_fwd = 2 * 4 * 16384 * 256 * 2 + 4 * 256 * 64 * 64 * 2
    assert f >= kernels_fwd + 2 * states
    assert b >= f + states
    q = P(B=1, H=4, T=16384 - 16, dk=256, dv=512)  # a ragged last chunk: not segmented
    assert L.gla_workspace_bytes(ctypes.byref(q), 0) < kernels_fwd + states


def test_segment_count_can_be_fixed(L):
    """GLA_SEGMENTS(n) overrides the shape's choice: 1 keeps every state on
    chip (no state arrays), T/C materializes every chunk's initial state (two
    [B H n d_k d_v] fp32 arrays in the forward's workspace, a third in the
    backward's); a count that does not divide T/C, a ragged T, too many heads
    or a segmented general form is refused."""
    seg = lambda n: n << gla.SEGMENTS_SHIFT
    long_ = dict(B=1, H=4, T=16384, dk=256, dv=512)
    auto = L.gla_workspace_bytes(ctypes.byref(P(**long_)), 0)
    one = L.gla_workspace_bytes(ctypes.byref(P(**long_, flags=seg(1))), 0)
    eight = L.gla_workspace_bytes(ctypes.byref(P(**long_, flags=seg(8))), 0)
    assert eight == auto  # the cost model's own choice for this shape
    state = 4 * 256 * 512 * 4  # one [B H d_k d_v] fp32 array
    for n in (2, 16, 256):
        f = L.gla_workspace_bytes(ctypes.byref(P(**long_, flags=seg(n))), 0)
        b = L.gla_workspace_bytes(ctypes.byref(P(**long_, flags=seg(n))), 1)
        assert 2 * n * state <= f - one < 2 * n * state + n * 4 * 256 * 4 + 3 * 256
        b1 = L.gla_workspace_bytes(ctypes.byref(P(**long_, flags=seg(1))), 1)
        assert 3 * n * state <= b - b1 < 3 * n * state + 2 * n * 4 * 256 * 4 + 4 * 256  # + decays, cST
    short = dict(T=256)  # N = 4 chunks of 64
    for n, ok in ((1, True), (2, True), (4, True), (3, False), (8, False)):
        p = P(**short, flags=seg(n))
        assert (L.gla_workspace_bytes(ctypes.byref(p), 1) > 0) == ok
        if not ok:  # (a valid problem would launch: never with these fake pointers)
            assert fwd_call(L, p) == gla.GLA_ERR_UNSUPPORTED
            assert bwd_call(L, p) == gla.GLA_ERR_UNSUPPORTED
    ragged = P(T=200, flags=seg(2))
    assert L.gla_workspace_bytes(ctypes.byref(ragged), 0) == 0
    assert fwd_call(L, ragged) == gla.GLA_ERR_UNSUPPORTED and bwd_call(L, ragged) == gla.GLA_ERR_UNSUPPORTED
    assert L.gla_workspace_bytes(ctypes.byref(P(T=200, flags=seg(1))), 0) > 0
    heads = P(B=1024, H=32, T=4096, flags=seg(2))  # 32768 heads x 2 segments > 65535
    assert L.gla_workspace_bytes(ctypes.byref(heads), 0) == 0
    assert fwd_call(L, heads) == gla.GLA_ERR_UNSUPPORTED
    # empty sequences accept any count; the general form only 0 and 1
    assert L.gla_workspace_bytes(ctypes.byref(P(T=0, flags=seg(3))), 1) >= 0
    assert L.gla_workspace_bytes(ctypes.byref(P(T=256, flags=seg(2))), 2) == 0
    assert L.gla_workspace_bytes(ctypes.byref(P(T=256, flags=seg(1))), 2) == \
        L.gla_workspace_bytes(ctypes.byref(P(T=256)), 2)
    args = (1, 1, 1, 1, 1, None, 1, None, 1, 1 << 40, None)
    assert L.gla_chunk_fwd_general(ctypes.byref(P(T=256, flags=seg(2))), *args) == gla.GLA_ERR_UNSUPPORTED
    assert L.gla_chunk_bwd_general(ctypes.byref(P(T=256, flags=seg(2))), 1, 1, 1, 1, 1, None, 1, 1, None, 1, 1, 1,
                                   1, 1, None, 1, 1 << 40, None) == gla.GLA_ERR_UNSUPPORTED


def fwd_call(L, p, ptr=1, ws=1, ws_bytes=1 << 40):
    return L.gla_chunk_fwd(ctypes.byref(p) if p is not None else None, ptr, ptr, ptr, ptr, None,
                           ptr, None, ws, ws_bytes, None)


def bwd_call(L, p, ptr=1, ws=1, ws_bytes=1 << 40):
    return L.gla_chunk_bwd(ctypes.byref(p), ptr, ptr, ptr, ptr, None, ptr, None, ptr, ptr, ptr,
                           ptr, None, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(io=7), gla.GLA_ERR_DTYPE),
    (dict(T=-1), gla.GLA_ERR_SHAPE),
    (dict(B=-2), gla.GLA_ERR_SHAPE),
    (dict(dk=0), gla.GLA_ERR_SHAPE),
    (dict(chunk=64, subchunk=48), gla.GLA_ERR_SHAPE),
    (dict(dk=24), gla.GLA_ERR_UNSUPPORTED),
    (dict(dk=272), gla.GLA_ERR_UNSUPPORTED),
    (dict(dv=2048), gla.GLA_ERR_UNSUPPORTED),
    (dict(chunk=128, subchunk=16), gla.GLA_ERR_UNSUPPORTED),
    (dict(chunk=64, subchunk=32), gla.GLA_ERR_UNSUPPORTED),
    (dict(io=gla.GLA_F32, dk=256), gla.GLA_ERR_UNSUPPORTED),
    (dict(B=65536, H=1), gla.GLA_ERR_UNSUPPORTED),
    (dict(B=256, H=256), gla.GLA_ERR_UNSUPPORTED),
    (dict(gate_tau=-16.0), gla.GLA_ERR_SHAPE),
    (dict(gate_tau=float("inf")), gla.GLA_ERR_SHAPE),
    (dict(gate_tau=float("nan")), gla.GLA_ERR_SHAPE),
])
def test_invalid_problems_are_rejected(L, kw, code):
    assert fwd_call(L, P(**kw)) == code
    assert bwd_call(L, P(**kw)) == code


def test_null_problem_and_pointers(L):
    assert fwd_call(L, None) == gla.GLA_ERR_NULL
    assert fwd_call(L, P(), ptr=None) == gla.GLA_ERR_NULL
    assert bwd_call(L, P(), ptr=None) == gla.GLA_ERR_NULL
    p = P()
    assert L.gla_recurrent_fwd(None, 1, 1, 1, 1, None, 1, None, None) == gla.GLA_ERR_NULL
    assert L.gla_recurrent_fwd(ctypes.byref(p), None, 1, 1, 1, None, 1, None, None) == gla.GLA_ERR_NULL


def test_general_form_entry_points_validate_like_the_others(L):
    p = P()
    args = lambda ptr: (ptr, ptr, ptr, ptr, ptr, None, ptr, None)
    assert L.gla_chunk_fwd_general(None, *args(1), 1, 1 << 40, None) == gla.GLA_ERR_NULL
    assert L.gla_chunk_fwd_general(ctypes.byref(P(dk=24)), *args(1), 1, 1 << 40, None) == gla.GLA_ERR_UNSUPPORTED
    assert L.gla_chunk_fwd_general(ctypes.byref(p), *args(None), 1, 1 << 40, None) == gla.GLA_ERR_NULL
    assert L.gla_chunk_fwd_general(ctypes.byref(p), *args(1), None, 0, None) == gla.GLA_ERR_WORKSPACE
    assert L.gla_recurrent_fwd_general(None, *args(1), None) == gla.GLA_ERR_NULL
    assert L.gla_recurrent_fwd_general(ctypes.byref(P(io=9)), *args(1), None) == gla.GLA_ERR_DTYPE
    assert L.gla_recurrent_fwd_general(ctypes.byref(p), *args(None), None) == gla.GLA_ERR_NULL
    # backward: log beta required, o required for dlog beta, the key-gate epilogue refused, op 2 workspace
    bw = lambda pp, lb=1, o=1, dlb=1, ws=1, nb=1 << 40: L.gla_chunk_bwd_general(
        ctypes.byref(pp), 1, 1, 1, 1, lb, None, o, 1, None, 1, 1, 1, 1, dlb, None, ws, nb, None)
    assert bw(p, lb=None) == gla.GLA_ERR_NULL
    assert bw(p, o=None) == gla.GLA_ERR_NULL
    assert bw(P(gate_tau=16.0)) == gla.GLA_ERR_UNSUPPORTED
    n1, n2 = L.gla_workspace_bytes(ctypes.byref(p), 1), L.gla_workspace_bytes(ctypes.byref(p), 2)
    assert n2 > n1 + 2 * 6 * 200 * 128 * 2
    assert bw(p, nb=n1) == gla.GLA_ERR_WORKSPACE
    assert L.gla_workspace_bytes(ctypes.byref(p), 3) == 0


def test_workspace_is_checked(L):
    p = P()
    need = L.gla_workspace_bytes(ctypes.byref(p), 0)
    assert fwd_call(L, p, ws=None) == gla.GLA_ERR_WORKSPACE
    assert fwd_call(L, p, ws_bytes=need - 1) == gla.GLA_ERR_WORKSPACE
    needb = L.gla_workspace_bytes(ctypes.byref(p), 1)
    assert bwd_call(L, p, ws_bytes=needb - 1) == gla.GLA_ERR_WORKSPACE


def test_empty_batch_needs_nothing(L):
    p = P(B=0)
    assert fwd_call(L, p, ptr=None, ws=None, ws_bytes=0) == gla.GLA_OK
    assert bwd_call(L, p, ptr=None, ws=None, ws_bytes=0) == gla.GLA_OK


def test_stage_selector_is_validated(L):
    assert fwd_call(L, P(flags=3 << 8)) == gla.GLA_ERR_SHAPE
    assert bwd_call(L, P(flags=6 << 8)) == gla.GLA_ERR_SHAPE
    assert fwd_call(L, P(B=0, flags=3 << 8), ptr=None, ws=None, ws_bytes=0) == gla.GLA_ERR_SHAPE


def og_fwd_call(L, p, eps=1e-5, ptr=1):
    return L.gla_output_gate_fwd(ctypes.byref(p) if p is not None else None, ptr, ptr, None, None,
                                 ctypes.c_float(eps), ptr, None, None)


def og_bwd_call(L, p, eps=1e-5, ptr=1, ws=1, ws_bytes=1 << 40):
    return L.gla_output_gate_bwd(ctypes.byref(p) if p is not None else None, ptr, ptr, None, None,
                                 ctypes.c_float(eps), ptr, ptr, ptr, ptr, ptr, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,eps,code", [
    (dict(io=7), 1e-5, gla.GLA_ERR_DTYPE),
    (dict(T=-1), 1e-5, gla.GLA_ERR_SHAPE),
    (dict(dv=0), 1e-5, gla.GLA_ERR_SHAPE),
    (dict(), 0.0, gla.GLA_ERR_SHAPE),
    (dict(), -1.0, gla.GLA_ERR_SHAPE),
    (dict(), float("nan"), gla.GLA_ERR_SHAPE),
    (dict(dv=24), 1e-5, gla.GLA_ERR_UNSUPPORTED),
    (dict(dv=2048), 1e-5, gla.GLA_ERR_UNSUPPORTED),
])
def test_output_gate_rejects_invalid_problems(L, kw, eps, code):
    assert og_fwd_call(L, P(**kw), eps) == code
    assert og_bwd_call(L, P(**kw), eps) == code


def test_output_gate_checks_pointers_and_workspace(L):
    L.gla_output_gate_workspace_bytes.restype = ctypes.c_size_t
    p = P()
    need = L.gla_output_gate_workspace_bytes(ctypes.byref(p))
    assert need == 2 * 3 * ((200 + 63) // 64) * 2 * 128 * 4
    assert og_fwd_call(L, None) == gla.GLA_ERR_NULL
    assert og_fwd_call(L, p, ptr=None) == gla.GLA_ERR_NULL
    assert og_bwd_call(L, p, ptr=None) == gla.GLA_ERR_NULL
    assert og_bwd_call(L, p, ws=None) == gla.GLA_ERR_WORKSPACE
    assert og_bwd_call(L, p, ws_bytes=need - 1) == gla.GLA_ERR_WORKSPACE
    assert og_fwd_call(L, P(B=0), ptr=None) == gla.GLA_OK


def test_noalloc_refuses_oversized_problems_before_any_launch(L):
    """gla_chunk_fwd_noalloc: a problem whose forward workspace exceeds the
    fixed scratch array gets GLA_ERR_SCRATCH without a HIP call (the dummy
    pointers are never touched); invalid problems get the forward's own
    validation errors."""
    p = P(B=64, H=4, T=4096, dk=256, dv=512)
    assert L.gla_workspace_bytes(ctypes.byref(p), 0) > gla.NOALLOC_SCRATCH_BYTES
    st = L.gla_chunk_fwd_noalloc(ctypes.byref(p), 16, 16, 16, None, None, 16, None, None)
    assert st == gla.GLA_ERR_SCRATCH
    assert L.gla_chunk_fwd_noalloc(None, 16, 16, 16, None, None, 16, None, None) == gla.GLA_ERR_NULL
    bad = P(dk=24)
    assert L.gla_chunk_fwd_noalloc(ctypes.byref(bad), 16, 16, 16, None, None, 16, None, None) == \
        gla.GLA_ERR_UNSUPPORTED
