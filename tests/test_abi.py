"""C-ABI checks that need no GPU: symbols, status strings, workspace sizes and
every argument check (they all run before the first HIP call, so only invalid
calls are made here -- a valid call would launch kernels)."""
import ctypes
import os
import re

import pytest

import paper_2607_14568_amd as gdn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gdn.h")

OK, INVALID, UNSUPPORTED, WORKSPACE, HIPERR = 0, 1, 2, 3, 4
A = 1 << 20          # a fake, 256-byte aligned "device address" (never dereferenced)


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(gdn.LIB_PATH):
        from paper_2607_14568_amd import build
        build.build_library(force=True)
    return gdn.lib()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gdn_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    names = _declared_functions()
    assert {"gdn_chunk_prefill", "gdn_decode_step", "gdn_chunk_prefill_workspace_bytes"} <= set(names)
    for name in names:
        assert hasattr(L, name), name


def test_version_and_status_strings(L):
    assert gdn.gdn_version() >= 1
    assert gdn.gdn_status_string(0) == "GDN_OK"
    assert gdn.gdn_status_string(3) == "GDN_ERR_WORKSPACE"
    assert gdn.gdn_status_string(99) == "unknown status"


def test_workspace_bytes():
    """The sequential plan's workspace: chunk terms per (chunk slot, head), and the ragged sequence table."""
    ws = gdn.gdn_chunk_prefill_workspace_bytes

    def seq(*a):
        return gdn.gdn_chunk_prefill_workspace_bytes_ex(*a, gdn.GDN_PLAN_SEQUENTIAL, 0)
    a = seq(1, 10240, 16, 128, 128, 64, 0, gdn.GDN_BF16)
    slots = 160 * 16
    assert a >= slots * (128 * 4 + 2 * 6 * 64 * 8 * 2)      # decay vectors + T, P fragments
    assert a % 256 == 0 and ws(1, 10240, 16, 128, 128, 64, 0, gdn.GDN_BF16) % 256 == 0
    assert seq(1, 10240, 16, 128, 128, 64, 0, gdn.GDN_F32) > a
    assert seq(1, 10241, 16, 128, 128, 64, 0, gdn.GDN_BF16) > a       # a partial chunk adds a slot
    assert seq(1, 20000, 16, 128, 128, 64, 8, gdn.GDN_BF16) > seq(1, 20000, 16, 128, 128, 64, 0, gdn.GDN_BF16)
    assert ws(1, 0, 16, 128, 128, 64, 0, gdn.GDN_BF16) == 0
    for bad in [(0, 10, 1, 64, 64, 64, 0, 0), (1, 10, 1, 96, 64, 64, 0, 0), (1, 10, 1, 64, 64, 48, 0, 0),
                (2, 10, 1, 64, 64, 64, 3, 0), (1, 10, 1, 64, 64, 64, 0, 7), (1, -1, 1, 64, 64, 64, 0, 0)]:
        assert ws(*bad) == 0, bad


def _plan(L, B, T, H, dk, dv, n_seqs, io, flags=0, segments=0, ws_bytes=None):
    """(form, segments) gdn_chunk_prefill_plan gives; with no device the automatic plan sees 0 CUs."""
    if ws_bytes is None:
        ws_bytes = L.gdn_chunk_prefill_workspace_bytes_ex(B, T, H, dk, dv, 64, n_seqs, io, flags, segments)
    form = ctypes.c_int(-1)
    n = L.gdn_chunk_prefill_plan(B, T, H, dk, dv, n_seqs, io, flags, segments, ws_bytes, None, ctypes.byref(form))
    return form.value, n


def test_plans_and_workspace():
    """The per-call plan (flags + segments) and the workspace each plan needs (pure host arithmetic; the
    workspace functions size the automatic plan for a 256-CU device)."""
    L = gdn.lib()
    ws, wsx = gdn.gdn_chunk_prefill_workspace_bytes, gdn.gdn_chunk_prefill_workspace_bytes_ex
    bf, f32 = gdn.GDN_BF16, gdn.GDN_F32
    SEQ, SEG, WIDE = gdn.GDN_PLAN_SEQUENTIAL, gdn.GDN_PLAN_SEGMENTED, gdn.GDN_PLAN_WIDE
    seq = {(io, H): wsx(1, 10240, H, 128, 128, 64, 0, io, SEQ, 0) for io in (bf, f32) for H in (1, 2, 4, 8, 16)}
    auto = {(io, H): ws(1, 10240, H, 128, 128, 64, 0, io) for io in (bf, f32) for H in (1, 2, 4, 8, 16)}
    # up to 8 heads split (the chain would leave most of 256 CUs idle; 8 bf16 heads take the wide form);
    # 16 heads stay sequential (the split forms' extra work outweighs the idle CUs they fill)
    for key in [(bf, 1), (bf, 2), (bf, 4), (bf, 8), (f32, 1), (f32, 2), (f32, 4), (f32, 8)]:
        assert auto[key] > seq[key], key
    assert auto[(f32, 16)] == seq[(f32, 16)] and auto[(bf, 16)] == seq[(bf, 16)]
    assert wsx(1, 10240, 16, 128, 128, 64, 0, bf, 0, 0) == auto[(bf, 16)]
    assert auto[(bf, 8)] == wsx(1, 10240, 8, 128, 128, 64, 0, bf, WIDE, 0)
    # short bf16 prompts stay sequential (the split's fixed costs outweigh its gain)
    assert ws(1, 2048, 2, 128, 128, 64, 0, bf) == wsx(1, 2048, 2, 128, 128, 64, 0, bf, SEQ, 0)
    # forced: more segments, more workspace; ragged input never splits
    two = wsx(1, 4096, 2, 128, 128, 64, 0, bf, SEG, 2)
    assert wsx(1, 4096, 2, 128, 128, 64, 0, bf, SEG, 8) > two
    rag = wsx(1, 4096, 2, 128, 128, 64, 3, bf, SEQ, 0)
    assert wsx(1, 4096, 2, 128, 128, 64, 3, bf, SEG, 8) == rag
    assert wsx(1, 4096, 4, 128, 128, 64, 0, bf, WIDE, 16) > wsx(1, 4096, 4, 128, 128, 64, 0, bf, WIDE, 4)
    # the plan a call takes: forced plans need no device
    assert _plan(L, 1, 10240, 16, 128, 128, 0, bf, WIDE) == (WIDE, 16)
    assert _plan(L, 1, 10240, 16, 128, 128, 0, bf, WIDE, 5) == (WIDE, 5)
    assert _plan(L, 1, 10240, 16, 64, 64, 0, bf, WIDE | gdn.GDN_GATE_LOGITS, 3) == (WIDE, 3)
    assert _plan(L, 1, 4096, 2, 128, 128, 0, bf, SEG, 3) == (SEG, 3)
    assert _plan(L, 1, 4096, 2, 128, 128, 3, bf, SEG, 3) == (SEQ, 1)      # ragged: sequential
    assert _plan(L, 1, 100, 2, 128, 128, 0, bf, SEG, 3) == (SEG, 2)       # two chunks: at most two segments
    assert _plan(L, 1, 64, 2, 128, 128, 0, bf, WIDE, 3) == (SEQ, 1)       # one chunk: nothing to split
    assert _plan(L, 1, 4096, 2, 128, 128, 0, bf, SEQ) == (SEQ, 1)
    assert _plan(L, 1, 4096, 2, 128, 128, 0, bf, 0, 1) == (SEQ, 1)
    # a workspace too small for the split: fewer segments, down to the sequential form
    small = wsx(1, 10240, 16, 128, 128, 64, 0, bf, SEQ, 0)
    assert _plan(L, 1, 10240, 16, 128, 128, 0, bf, WIDE, 8, ws_bytes=small) == (SEQ, 1)
    mid = wsx(1, 10240, 16, 128, 128, 64, 0, bf, WIDE, 4)
    assert _plan(L, 1, 10240, 16, 128, 128, 0, bf, WIDE, 8, ws_bytes=mid) == (WIDE, 4)
    # rejected: the wide form needs dense bf16 input with dk == dv and no key normalisation; one plan at a
    # time; segment counts only with a segmented plan and within 0..64; bad sizes
    for bad in [(1, 4096, 2, 128, 128, 0, f32, WIDE, 0), (1, 4096, 2, 128, 128, 3, bf, WIDE, 0),
                (1, 4096, 2, 128, 64, 0, bf, WIDE, 0), (1, 4096, 2, 128, 128, 0, bf, WIDE | gdn.GDN_QK_L2NORM, 0),
                (1, 4096, 2, 128, 128, 0, bf, SEG | WIDE, 0), (1, 4096, 2, 128, 128, 0, bf, 0, 3),
                (1, 4096, 2, 128, 128, 0, bf, SEQ, 3), (1, 4096, 2, 128, 128, 0, bf, SEG, 65),
                (1, 4096, 2, 128, 128, 0, bf, SEG, -1), (1, 4096, 2, 128, 128, 0, bf, 128, 0),
                (0, 10, 1, 64, 64, 0, bf, 0, 0), (1, 10, 1, 96, 64, 0, bf, 0, 0), (2, 10, 1, 64, 64, 3, bf, 0, 0),
                (1, 10, 1, 64, 64, 0, 7, 0, 0)]:
        assert _plan(L, *bad, ws_bytes=1 << 40) == (0, 0), bad
        assert wsx(bad[0], bad[1], bad[2], bad[3], bad[4], 64, bad[5], bad[6], bad[7], bad[8]) == 0, bad


def _prefill(L, **kw):
    a = dict(q=A, k=A, v=A, g=A, beta=A, S0=None, o=A, ST=A, B=1, T=128, H=2, dk=64, dv=64, chunk=64,
             cu=None, n_seqs=0, io=0, scale=1.0, ws=A, ws_bytes=1 << 40, stream=None)
    a.update(kw)
    return L.gdn_chunk_prefill(a["q"], a["k"], a["v"], a["g"], a["beta"], a["S0"], a["o"], a["ST"],
                               a["B"], a["T"], a["H"], a["dk"], a["dv"], a["chunk"], a["cu"], a["n_seqs"],
                               a["io"], a["scale"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(io=2), INVALID),
    (dict(io=-1), INVALID),
    (dict(B=0), INVALID),
    (dict(H=0), INVALID),
    (dict(T=-5), INVALID),
    (dict(dk=0), INVALID),
    (dict(dk=96), UNSUPPORTED),
    (dict(dv=256), UNSUPPORTED),
    (dict(dk=32, dv=32), UNSUPPORTED),
    (dict(H=1 << 19), UNSUPPORTED),
    (dict(chunk=0), INVALID),
    (dict(chunk=48), UNSUPPORTED),
    (dict(chunk=256), UNSUPPORTED),
    (dict(q=None), INVALID),
    (dict(k=None), INVALID),
    (dict(v=None), INVALID),
    (dict(g=None), INVALID),
    (dict(beta=None), INVALID),
    (dict(o=None), INVALID),
    (dict(q=A + 8), INVALID),
    (dict(S0=A + 4), INVALID),
    (dict(ST=A + 2), INVALID),
    (dict(cu=A), INVALID),                       # cu_seqlens without n_seqs
    (dict(n_seqs=3), INVALID),                   # n_seqs without cu_seqlens
    (dict(cu=A, n_seqs=2, B=2), INVALID),        # ragged needs B == 1
    (dict(cu=A + 2, n_seqs=2), INVALID),         # misaligned offsets
    (dict(g=A + 2), INVALID),
    (dict(beta=A + 1), INVALID),
    (dict(v=A + 4), INVALID),
    (dict(o=A + 8), INVALID),
    (dict(n_seqs=-1, cu=A), INVALID),
    (dict(ws=None), WORKSPACE),
    (dict(ws_bytes=1000), WORKSPACE),
    (dict(ws=A + 16), INVALID),                  # workspace not 256-byte aligned
])
def test_prefill_argument_checks(L, kw, code):
    rc = _prefill(L, **kw)
    assert rc == code, (kw, rc, L.gdn_last_error_message())
    assert L.gdn_last_error_message().decode()


def _snapshots(L, snap_every=1, snaps=A, **kw):
    a = dict(q=A, k=A, v=A, g=A, beta=A, S0=None, o=A, ST=A, B=1, T=128, H=2, dk=64, dv=64, chunk=64,
             cu=None, n_seqs=0, io=0, scale=1.0, ws=A, ws_bytes=1 << 40, stream=None)
    a.update(kw)
    return L.gdn_chunk_prefill_snapshots(a["q"], a["k"], a["v"], a["g"], a["beta"], a["S0"], a["o"], a["ST"],
                                         a["B"], a["T"], a["H"], a["dk"], a["dv"], a["chunk"], a["cu"], a["n_seqs"],
                                         a["io"], a["scale"], snap_every, snaps, a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(snap_every=0), INVALID),
    (dict(snap_every=-3), INVALID),
    (dict(snaps=None), INVALID),              # T=128: one snapshot falls inside the prompt
    (dict(snaps=A + 8), INVALID),             # not 16-byte aligned
    (dict(snaps=A, chunk=32), UNSUPPORTED),   # the prefill's own checks still apply
    (dict(snaps=A, io=5), INVALID),
    (dict(snaps=A, ws_bytes=100), WORKSPACE),
])
def test_snapshot_argument_checks(L, kw, code):
    rc = _snapshots(L, **kw)
    assert rc == code, (kw, rc, L.gdn_last_error_message())
    assert L.gdn_last_error_message().decode()


def test_prefill_workspace_exact_boundary(L):
    need = gdn.gdn_chunk_prefill_workspace_bytes(1, 128, 2, 64, 64, 64, 0, 0)
    assert _prefill(L, ws_bytes=need - 1) == WORKSPACE


def _prefill_grouped(L, **kw):
    a = dict(q=A, k=A, v=A, g=A, beta=A, S0=None, o=A, ST=A, B=1, T=128, H=4, Hk=2, dk=64, dv=64, chunk=64,
             cu=None, n_seqs=0, io=0, scale=1.0, ws=A, ws_bytes=1 << 40, stream=None)
    a.update(kw)
    return L.gdn_chunk_prefill_grouped(a["q"], a["k"], a["v"], a["g"], a["beta"], a["S0"], a["o"], a["ST"],
                                       a["B"], a["T"], a["H"], a["Hk"], a["dk"], a["dv"], a["chunk"], a["cu"],
                                       a["n_seqs"], a["io"], a["scale"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(Hk=0), INVALID),
    (dict(Hk=-2), INVALID),
    (dict(Hk=8), INVALID),                    # more key heads than value heads
    (dict(Hk=3), INVALID),                    # does not divide H = 4
    (dict(H=6, Hk=4), INVALID),
    (dict(H=0, Hk=1), INVALID),
    (dict(dk=96), UNSUPPORTED),               # the prefill's own checks still apply
    (dict(chunk=48), UNSUPPORTED),
    (dict(q=A + 8), INVALID),
    (dict(ws_bytes=1000), WORKSPACE),
])
def test_grouped_prefill_argument_checks(L, kw, code):
    rc = _prefill_grouped(L, **kw)
    assert rc == code, (kw, rc, L.gdn_last_error_message())
    assert L.gdn_last_error_message().decode()


def _decode_grouped(L, **kw):
    a = dict(q=A, k=A, v=A, g=A, beta=A, S=A, o=A, B=4, H=4, Hk=2, dk=128, dv=128, io=0, scale=1.0, stream=None)
    a.update(kw)
    return L.gdn_decode_step_grouped(a["q"], a["k"], a["v"], a["g"], a["beta"], a["S"], a["o"], a["B"], a["H"],
                                     a["Hk"], a["dk"], a["dv"], a["io"], a["scale"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(Hk=0), INVALID), (dict(Hk=3), INVALID), (dict(Hk=5), INVALID), (dict(B=0), INVALID),
    (dict(dk=100), UNSUPPORTED), (dict(S=None), INVALID), (dict(S=A + 8), INVALID),
])
def test_grouped_decode_argument_checks(L, kw, code):
    assert _decode_grouped(L, **kw) == code


def test_binding_grouped_shapes():
    import torch
    if torch.cuda.is_available():
        pytest.skip("checks CPU-tensor rejection only")
    x = torch.zeros(1, 4, 2, 64)
    v = torch.zeros(1, 4, 4, 64)
    g = torch.zeros(1, 4, 4)
    with pytest.raises(TypeError):
        gdn.gdn_chunk_prefill_grouped(x, x, v, g, g)
    with pytest.raises(TypeError):
        gdn.gdn_decode_step_grouped(x[0], x[0], v[0], g[0], g[0], torch.zeros(1, 4, 64, 64))


def _prefill_ex(L, **kw):
    a = dict(q=A, k=A, v=A, g=A, beta=A, S0=None, o=A, ST=A, B=1, T=128, H=4, Hk=2, dk=64, dv=64, chunk=64,
             cu=None, n_seqs=0, io=0, scale=1.0, flags=3, segments=0, ws=A, ws_bytes=1 << 40, stream=None)
    a.update(kw)
    return L.gdn_chunk_prefill_ex(a["q"], a["k"], a["v"], a["g"], a["beta"], a["S0"], a["o"], a["ST"],
                                  a["B"], a["T"], a["H"], a["Hk"], a["dk"], a["dv"], a["chunk"], a["cu"],
                                  a["n_seqs"], a["io"], a["scale"], a["flags"], a["segments"], a["ws"], a["ws_bytes"],
                                  a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(flags=4), INVALID), (dict(flags=-1), INVALID), (dict(flags=8 | 1), INVALID),
    (dict(flags=16 | 32), INVALID), (dict(flags=32 | 64), INVALID), (dict(flags=128), INVALID),
    (dict(segments=-1), INVALID), (dict(segments=65), INVALID), (dict(segments=4), INVALID),
    (dict(flags=16, segments=4), INVALID),
    (dict(flags=64, io=0), UNSUPPORTED), (dict(flags=64 | 1, io=1), UNSUPPORTED), (dict(flags=64, io=1, dv=128),
                                                                                   UNSUPPORTED),
    (dict(Hk=3), INVALID), (dict(dk=96), UNSUPPORTED), (dict(chunk=96), UNSUPPORTED),
    (dict(chunk=32, flags=32), UNSUPPORTED), (dict(chunk=128, flags=64, io=1, dk=128, dv=128), UNSUPPORTED),
    (dict(chunk=16, flags=16, segments=2), INVALID),
    (dict(q=None), INVALID), (dict(ws_bytes=10), WORKSPACE), (dict(io=7), INVALID),
])
def test_ex_prefill_argument_checks(L, kw, code):
    rc = _prefill_ex(L, **kw)
    assert rc == code, (kw, rc, L.gdn_last_error_message())
    assert L.gdn_last_error_message().decode()


@pytest.mark.parametrize("kw,code", [
    (dict(flags=4), INVALID), (dict(flags=-2), INVALID), (dict(Hk=3), INVALID), (dict(dk=100), UNSUPPORTED),
    (dict(S=None), INVALID),
])
def test_ex_decode_argument_checks(L, kw, code):
    a = dict(q=A, k=A, v=A, g=A, beta=A, S=A, o=A, B=4, H=4, Hk=2, dk=128, dv=128, io=0, scale=1.0, flags=1,
             stream=None)
    a.update(kw)
    rc = L.gdn_decode_step_ex(a["q"], a["k"], a["v"], a["g"], a["beta"], a["S"], a["o"], a["B"], a["H"], a["Hk"],
                              a["dk"], a["dv"], a["io"], a["scale"], a["flags"], a["stream"])
    assert rc == code, (kw, rc)


@pytest.mark.parametrize("kw,code", [
    (dict(io=2), INVALID), (dict(io=0), UNSUPPORTED), (dict(B=0), INVALID), (dict(T=-1), INVALID),
    (dict(H=0), INVALID), (dict(Hkv=0), INVALID), (dict(Hkv=3), INVALID), (dict(Hkv=8), INVALID),
    (dict(d=0), INVALID), (dict(d=96), UNSUPPORTED), (dict(d=256), UNSUPPORTED),
    (dict(q=None), INVALID), (dict(o=None), INVALID), (dict(k=A + 8), INVALID), (dict(v=A + 2), INVALID),
    (dict(H=1 << 14), UNSUPPORTED),
    (dict(cu=A), INVALID),                       # cu_seqlens without n_seqs
    (dict(n=3), INVALID),                        # n_seqs without cu_seqlens
    (dict(cu=A, n=2, B=2), INVALID),             # packed sequences need B == 1
    (dict(cu=A + 2, n=2), INVALID),              # misaligned offsets
    (dict(cu=A, n=-1), INVALID),
])
def test_attention_argument_checks(L, kw, code):
    a = dict(q=A, k=A, v=A, o=A, B=1, T=256, H=4, Hkv=2, d=128, cu=None, n=0, io=1, scale=0.088, stream=None)
    a.update(kw)
    rc = L.gdn_attention_prefill(a["q"], a["k"], a["v"], a["o"], a["B"], a["T"], a["H"], a["Hkv"], a["d"], a["cu"],
                                 a["n"], a["io"], a["scale"], a["stream"])
    assert rc == code, (kw, rc, L.gdn_last_error_message())


def test_attention_empty_prompt_is_a_no_op(L):
    assert L.gdn_attention_prefill(None, None, None, None, 2, 0, 4, 2, 128, None, 0, 1, 0.1, None) == OK


def test_snapshots_ex_argument_checks(L):
    def call(**kw):
        a = dict(Hk=2, flags=3, snap_every=1, snaps=A, chunk=64, ws_bytes=1 << 40)
        a.update(kw)
        return L.gdn_chunk_prefill_snapshots_ex(A, A, A, A, A, None, A, A, 1, 128, 4, a["Hk"], 64, 64, a["chunk"], None,
                                                0, 0, 1.0, a["flags"], a["snap_every"], a["snaps"], A, a["ws_bytes"],
                                                None)
    assert call(snap_every=0) == INVALID
    assert call(snaps=None) == INVALID
    assert call(flags=4) == INVALID
    assert call(flags=16) == INVALID           # snapshots take no plan
    assert call(flags=64) == INVALID
    assert call(Hk=3) == INVALID
    assert call(chunk=32) == UNSUPPORTED
    assert call(ws_bytes=100) == WORKSPACE


def _decode(L, **kw):
    a = dict(q=A, k=A, v=A, g=A, beta=A, S=A, o=A, B=4, H=2, dk=128, dv=128, io=0, scale=1.0, stream=None)
    a.update(kw)
    return L.gdn_decode_step(a["q"], a["k"], a["v"], a["g"], a["beta"], a["S"], a["o"], a["B"], a["H"],
                             a["dk"], a["dv"], a["io"], a["scale"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(io=3), INVALID), (dict(B=0), INVALID), (dict(H=-1), INVALID),
    (dict(dk=100), UNSUPPORTED), (dict(dv=32), UNSUPPORTED), (dict(dk=0), INVALID),
    (dict(q=None), INVALID), (dict(S=None), INVALID), (dict(o=None), INVALID),
    (dict(g=None), INVALID), (dict(v=A + 2), INVALID), (dict(S=A + 8), INVALID),
    (dict(g=A + 2), INVALID), (dict(q=A + 1, io=1), INVALID),
])
def test_decode_argument_checks(L, kw, code):
    assert _decode(L, **kw) == code


def test_binding_rejects_cpu_tensors():
    import torch
    x = torch.zeros(1, 4, 1, 64)
    g = torch.zeros(1, 4, 1)
    with pytest.raises(TypeError):
        gdn.gdn_chunk_prefill(x, x, x, g, g)
    with pytest.raises(TypeError):
        gdn.gdn_decode_step(x[0], x[0], x[0], g[0], g[0], torch.zeros(1, 4, 64, 64))


def test_product_package_does_not_reach_the_oracle():
    """The HIP path never imports or calls the oracle (no CPU fallback)."""
    pkg = os.path.join(ROOT, "paper_2607_14568_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".cpp", ".h")) and fn != "inputs.py":
                text = open(os.path.join(dirpath, fn)).read()
                assert "oracle" not in text, fn
    assert "import oracle" not in open(os.path.join(pkg, "inputs.py")).read()


def test_generic_chunk_workspace():
    """Chunk lengths 16, 32 and 128 take the generic path: per (chunk slot, head) 4 C floats and two C x C fp32
    matrices after the status word (and the ragged table), sequential plan only."""
    wsx = gdn.gdn_chunk_prefill_workspace_bytes_ex
    bf, f32 = gdn.GDN_BF16, gdn.GDN_F32
    rnd = lambda x: (x + 255) // 256 * 256
    for C in (16, 32, 128):
        for T, H in ((10240, 16), (1000, 3), (1, 1), (C, 2), (C + 1, 2)):
            items = -(-T // C) * H
            want = 256 + rnd(items * 4 * C * 4) + 2 * rnd(items * C * C * 4)
            for io in (bf, f32):
                assert wsx(1, T, H, 128, 128, C, 0, io, 0, 0) == want, (C, T, H)
                assert wsx(1, T, H, 64, 64, C, 0, io, gdn.GDN_PLAN_SEQUENTIAL, 0) == want
        assert gdn.gdn_chunk_prefill_workspace_bytes(1, 0, 4, 128, 128, C, 0, bf) == 0
        cpt = -(-1000 // C)
        items = (cpt + 3) * 2
        table = rnd((4 * 4 + 2 * (cpt + 2)) * 4)
        assert wsx(1, 1000, 2, 128, 128, C, 3, bf, 0, 0) == 256 + table + rnd(items * 4 * C * 4) + 2 * rnd(
            items * C * C * 4)
        for fl, seg in ((gdn.GDN_PLAN_SEGMENTED, 0), (gdn.GDN_PLAN_WIDE, 0), (gdn.GDN_PLAN_SEGMENTED, 4)):
            assert wsx(1, 1000, 2, 128, 128, C, 0, bf, fl, seg) == 0, (C, fl, seg)
    for bad in (0, 8, 48, 96, 256):
        assert wsx(1, 1000, 2, 128, 128, bad, 0, bf, 0, 0) == 0, bad
