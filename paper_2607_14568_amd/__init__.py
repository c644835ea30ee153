"""Gated delta-rule prefill and decode on MI355X (gfx950).

A thin ctypes binding over ``libgdn.so`` (C ABI in ``include/gdn.h``).  The
functions carry the C names and only marshal arguments: every step of the
computation runs in the library's HIP kernels.  PyTorch supplies device memory
and the current stream.  There is no CPU fallback: if the library is not built
or no GPU is present, calls raise.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "GDN_F32", "GDN_BF16", "GdnError", "lib", "gdn_version", "gdn_status_string",
    "gdn_chunk_prefill_workspace_bytes", "gdn_chunk_prefill_workspace_bytes_ex", "gdn_chunk_prefill",
    "gdn_decode_step", "gdn_chunk_prefill_plan", "gdn_chunk_prefill_snapshots",
    "GDN_PLAN_SEQUENTIAL", "GDN_PLAN_SEGMENTED", "GDN_PLAN_WIDE",
    "gdn_chunk_prefill_grouped", "gdn_decode_step_grouped", "gdn_chunk_prefill_ex", "gdn_decode_step_ex",
    "GDN_QK_L2NORM", "GDN_GATE_LOGITS", "gdn_attention_prefill", "gdn_chunk_prefill_snapshots_ex",
    "gdn_workspace_status", "GDN_ERR_WAIT", "GDN_TEST_WITHHOLD",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgdn.so")

GDN_F32, GDN_BF16 = 0, 1
GDN_QK_L2NORM, GDN_GATE_LOGITS = 1, 2
GDN_PLAN_SEQUENTIAL, GDN_PLAN_SEGMENTED, GDN_PLAN_WIDE = 16, 32, 64
GDN_TEST_WITHHOLD = 256
GDN_ERR_WAIT = 5
_IO = {torch.float32: GDN_F32, torch.bfloat16: GDN_BF16}
_lib = None


class GdnError(RuntimeError):
    def __init__(self, status, message):
        super().__init__("%s: %s" % (gdn_status_string(status), message))
        self.status = status


def lib():
    """The loaded ``libgdn.so`` (ctypes.CDLL) with argument types declared."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libgdn.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P, I, F, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
        L.gdn_version.restype = I
        L.gdn_status_string.argtypes = [I]
        L.gdn_status_string.restype = ctypes.c_char_p
        L.gdn_last_error_message.restype = ctypes.c_char_p
        L.gdn_chunk_prefill_workspace_bytes.argtypes = [I, I, I, I, I, I, I, I]
        L.gdn_chunk_prefill_workspace_bytes.restype = S
        L.gdn_chunk_prefill_workspace_bytes_ex.argtypes = [I] * 10
        L.gdn_chunk_prefill_workspace_bytes_ex.restype = S
        L.gdn_chunk_prefill.argtypes = [P, P, P, P, P, P, P, P, I, I, I, I, I, I, P, I, I, F, P, S, P]
        L.gdn_chunk_prefill.restype = I
        L.gdn_chunk_prefill_grouped.argtypes = [P, P, P, P, P, P, P, P, I, I, I, I, I, I, I, P, I, I, F, P, S, P]
        L.gdn_chunk_prefill_grouped.restype = I
        L.gdn_chunk_prefill_ex.argtypes = [P, P, P, P, P, P, P, P, I, I, I, I, I, I, I, P, I, I, F, I, I, P, S, P]
        L.gdn_chunk_prefill_ex.restype = I
        L.gdn_chunk_prefill_snapshots.argtypes = [P, P, P, P, P, P, P, P, I, I, I, I, I, I, P, I, I, F, I, P, P, S,
                                                  P]
        L.gdn_chunk_prefill_snapshots.restype = I
        L.gdn_chunk_prefill_snapshots_ex.argtypes = [P, P, P, P, P, P, P, P, I, I, I, I, I, I, I, P, I, I, F, I, I, P, P,
                                                     S, P]
        L.gdn_chunk_prefill_snapshots_ex.restype = I
        L.gdn_chunk_prefill_noalloc.argtypes = [P, P, P, P, P, P, P, P, I, I, I, I, I, I, I, P, I, I, F, I, I, P]
        L.gdn_chunk_prefill_noalloc.restype = I
        L.gdn_chunk_prefill_plan.argtypes = [I, I, I, I, I, I, I, I, I, S, P, ctypes.POINTER(I)]
        L.gdn_chunk_prefill_plan.restype = I
        L.gdn_decode_step.argtypes = [P, P, P, P, P, P, P, I, I, I, I, I, F, P]
        L.gdn_decode_step.restype = I
        L.gdn_decode_step_grouped.argtypes = [P, P, P, P, P, P, P, I, I, I, I, I, I, F, P]
        L.gdn_decode_step_grouped.restype = I
        L.gdn_decode_step_ex.argtypes = [P, P, P, P, P, P, P, I, I, I, I, I, I, F, I, P]
        L.gdn_decode_step_ex.restype = I
        L.gdn_attention_prefill.argtypes = [P, P, P, P, I, I, I, I, I, P, I, I, F, P]
        L.gdn_attention_prefill.restype = I
        L.gdn_workspace_status.argtypes = [P, S, P]
        L.gdn_workspace_status.restype = I
        _lib = L
    return _lib


def gdn_version() -> int:
    return int(lib().gdn_version())


def gdn_status_string(status: int) -> str:
    return lib().gdn_status_string(int(status)).decode()


def _check(status):
    if status != 0:
        raise GdnError(status, lib().gdn_last_error_message().decode())


def gdn_workspace_status(workspace=None, device=None):
    """Waits for the current stream and raises GdnError(GDN_ERR_WAIT) if a one-launch prefill on ``workspace``
    (a uint8 CUDA tensor; None: the scratch of ``gdn_chunk_prefill_noalloc``) gave up waiting for its chunk terms
    since the last check (the word is then cleared)."""
    if workspace is None:
        dev = torch.device("cuda", torch.cuda.current_device() if device is None else device)
        _check(lib().gdn_workspace_status(None, 0, _stream(dev)))
    else:
        _dev(workspace, "workspace")
        _check(lib().gdn_workspace_status(_ptr(workspace), workspace.numel() * workspace.element_size(),
                                          _stream(workspace.device)))


def gdn_chunk_prefill_workspace_bytes(B, T, H, dk, dv, chunk=64, n_seqs=0, io_dtype=GDN_BF16) -> int:
    return int(lib().gdn_chunk_prefill_workspace_bytes(B, T, H, dk, dv, chunk, n_seqs, io_dtype))


def gdn_chunk_prefill_workspace_bytes_ex(B, T, H, dk, dv, chunk=64, n_seqs=0, io_dtype=GDN_BF16, flags=0,
                                         segments=0) -> int:
    return int(lib().gdn_chunk_prefill_workspace_bytes_ex(B, T, H, dk, dv, chunk, n_seqs, io_dtype, int(flags),
                                                          int(segments)))


def gdn_chunk_prefill_plan(B, T, H, dk, dv, n_seqs=0, io_dtype=GDN_BF16, flags=0, segments=0,
                           workspace_bytes=None, device=None):
    """``(form, segments)`` a prefill of these sizes would take on ``device`` (form: a GDN_PLAN_* bit).

    ``workspace_bytes`` defaults to what ``gdn_chunk_prefill_workspace_bytes_ex`` gives.
    """
    if workspace_bytes is None:
        workspace_bytes = gdn_chunk_prefill_workspace_bytes_ex(B, T, H, dk, dv, 64, n_seqs, io_dtype, flags, segments)
    form = ctypes.c_int(0)
    stream = _stream(torch.device("cuda", torch.cuda.current_device() if device is None else device))
    n = int(lib().gdn_chunk_prefill_plan(B, T, H, dk, dv, n_seqs, io_dtype, int(flags), int(segments),
                                         int(workspace_bytes), stream, ctypes.byref(form)))
    return int(form.value), n


def _dev(t, name, dtype=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("%s must be a CUDA (HIP) tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    return t


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _prefill_args(q, k, v, g, beta, S0, chunk, cu_seqlens, o, S_T, store_state, workspace, grouped=False, flags=0,
                  segments=0, with_workspace=True):
    if q.dtype not in _IO:
        raise TypeError("q must be float32 or bfloat16")
    io = _IO[q.dtype]
    for name, t in (("q", q), ("k", k), ("v", v)):
        _dev(t, name, q.dtype)
    _dev(g, "g", torch.float32)
    _dev(beta, "beta", torch.float32)
    B, T, HK, dk = q.shape
    H = v.shape[2] if grouped else HK
    dv = v.shape[-1]
    if k.shape != q.shape or tuple(v.shape[:3]) != (B, T, H) or tuple(g.shape) != (B, T, H) \
            or beta.shape != g.shape:
        raise ValueError("inconsistent shapes q%s k%s v%s g%s beta%s" % (
            tuple(q.shape), tuple(k.shape), tuple(v.shape), tuple(g.shape), tuple(beta.shape)))
    n_seqs = 0
    if cu_seqlens is not None:
        _dev(cu_seqlens, "cu_seqlens", torch.int32)
        n_seqs = cu_seqlens.numel() - 1
    n = n_seqs if n_seqs else B
    if S0 is not None:
        _dev(S0, "S0", torch.float32)
        if tuple(S0.shape) != (n, H, dv, dk):
            raise ValueError("S0 must be [%d,%d,%d,%d]" % (n, H, dv, dk))
    if o is None:
        o = torch.empty_like(v)
    else:
        _dev(o, "o", q.dtype)
    if store_state and S_T is None:
        S_T = torch.empty((n, H, dv, dk), device=q.device, dtype=torch.float32)
    elif S_T is not None:
        _dev(S_T, "S_T", torch.float32)
    if not with_workspace:
        return dict(io=io, B=B, T=T, H=H, HK=HK, dk=dk, dv=dv, n=n, n_seqs=n_seqs, o=o, S_T=S_T)
    need = gdn_chunk_prefill_workspace_bytes_ex(B, T, H, dk, dv, chunk, n_seqs, io, flags, segments)
    if workspace is None:
        workspace = torch.empty(max(need, 1), device=q.device, dtype=torch.uint8)
    return dict(io=io, B=B, T=T, H=H, HK=HK, dk=dk, dv=dv, n=n, n_seqs=n_seqs, o=o, S_T=S_T, workspace=workspace)


def gdn_chunk_prefill(q, k, v, g, beta, S0=None, *, chunk=64, cu_seqlens=None, scale=1.0,
                      o=None, S_T=None, store_state=True, workspace=None):
    """Chunked prefill; see ``gdn_chunk_prefill`` in include/gdn.h.

    q,k [B,T,H,dk] and v [B,T,H,dv] (fp32 or bf16, same dtype); g, beta [B,T,H]
    fp32; S0 [n,H,dv,dk] fp32 or None.  Ragged: B == 1 and ``cu_seqlens`` an
    int32 CUDA tensor [n+1].  Returns ``(o, S_T)`` (S_T is None when
    ``store_state`` is False).  ``S_T`` may be passed (also ``S_T is S0``).
    """
    a = _prefill_args(q, k, v, g, beta, S0, chunk, cu_seqlens, o, S_T, store_state, workspace)
    _check(lib().gdn_chunk_prefill(
        _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S0), _ptr(a["o"]), _ptr(a["S_T"]),
        a["B"], a["T"], a["H"], a["dk"], a["dv"], chunk, _ptr(cu_seqlens), a["n_seqs"], a["io"], float(scale),
        _ptr(a["workspace"]), a["workspace"].numel(), _stream(q.device)))
    return a["o"], a["S_T"]


def gdn_chunk_prefill_grouped(q, k, v, g, beta, S0=None, *, chunk=64, cu_seqlens=None, scale=1.0,
                              o=None, S_T=None, store_state=True, workspace=None):
    """Prefill with grouped key heads; see ``gdn_chunk_prefill_grouped`` in include/gdn.h.

    q,k [B,T,H_k,dk]; v [B,T,H,dv]; g, beta [B,T,H]; value head h reads key head
    h // (H // H_k).  Otherwise as ``gdn_chunk_prefill``.
    """
    a = _prefill_args(q, k, v, g, beta, S0, chunk, cu_seqlens, o, S_T, store_state, workspace, grouped=True)
    _check(lib().gdn_chunk_prefill_grouped(
        _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S0), _ptr(a["o"]), _ptr(a["S_T"]),
        a["B"], a["T"], a["H"], a["HK"], a["dk"], a["dv"], chunk, _ptr(cu_seqlens), a["n_seqs"], a["io"],
        float(scale), _ptr(a["workspace"]), a["workspace"].numel(), _stream(q.device)))
    return a["o"], a["S_T"]


def gdn_chunk_prefill_ex(q, k, v, g, beta, S0=None, *, flags=0, segments=0, chunk=64, cu_seqlens=None, scale=1.0,
                         o=None, S_T=None, store_state=True, workspace=None):
    """Prefill with in-kernel input transforms and a per-call plan; see ``gdn_chunk_prefill_ex`` in include/gdn.h.

    Shapes as ``gdn_chunk_prefill_grouped``.  ``flags``: GDN_QK_L2NORM (q, k taken
    unnormalised) and/or GDN_GATE_LOGITS (``g``, ``beta`` hold the logits a, b), and at
    most one of GDN_PLAN_SEQUENTIAL, GDN_PLAN_SEGMENTED, GDN_PLAN_WIDE; ``segments``
    the segments per sequence of a segmented plan (0: the plan's own count).
    """
    a = _prefill_args(q, k, v, g, beta, S0, chunk, cu_seqlens, o, S_T, store_state, workspace, grouped=True,
                      flags=flags, segments=segments)
    _check(lib().gdn_chunk_prefill_ex(
        _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S0), _ptr(a["o"]), _ptr(a["S_T"]),
        a["B"], a["T"], a["H"], a["HK"], a["dk"], a["dv"], chunk, _ptr(cu_seqlens), a["n_seqs"], a["io"],
        float(scale), int(flags), int(segments), _ptr(a["workspace"]), a["workspace"].numel(), _stream(q.device)))
    return a["o"], a["S_T"]


GDN_NOALLOC_SCRATCH_BYTES = 64 << 20


def gdn_chunk_prefill_noalloc(q, k, v, g, beta, S0=None, *, flags=0, segments=0, chunk=64, cu_seqlens=None,
                              scale=1.0, o=None, S_T=None, store_state=True):
    """``gdn_chunk_prefill_ex`` on the library's own per-device scratch (no workspace, no device
    allocation inside the call); see ``gdn_chunk_prefill_noalloc`` in include/gdn.h.  Pass ``o``
    (and ``S_T``, or ``store_state=False``) to allocate nothing here either."""
    a = _prefill_args(q, k, v, g, beta, S0, chunk, cu_seqlens, o, S_T, store_state, None, grouped=True,
                      flags=flags, segments=segments, with_workspace=False)
    _check(lib().gdn_chunk_prefill_noalloc(
        _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S0), _ptr(a["o"]), _ptr(a["S_T"]),
        a["B"], a["T"], a["H"], a["HK"], a["dk"], a["dv"], chunk, _ptr(cu_seqlens), a["n_seqs"], a["io"],
        float(scale), int(flags), int(segments), _stream(q.device)))
    return a["o"], a["S_T"]


def gdn_chunk_prefill_snapshots(q, k, v, g, beta, S0=None, *, snap_every, chunk=64, cu_seqlens=None, scale=1.0,
                                o=None, S_T=None, snaps=None, store_state=True, workspace=None):
    """Prefill that also returns state snapshots; see ``gdn_chunk_prefill_snapshots`` in include/gdn.h.

    Returns ``(o, S_T, snaps)``; ``snaps`` is [n, (T-1) // (snap_every*chunk), H, dv, dk] fp32
    (allocated zero-filled when not given; entries past a sequence's last snapshot keep their values).
    """
    a = _prefill_args(q, k, v, g, beta, S0, chunk, cu_seqlens, o, S_T, store_state, workspace)
    n_snap = max(0, (a["T"] - 1) // (int(snap_every) * chunk)) if snap_every >= 1 else 0
    shape = (a["n"], n_snap, a["H"], a["dv"], a["dk"])
    if snaps is None:
        snaps = torch.zeros(shape, device=q.device, dtype=torch.float32)
    else:
        _dev(snaps, "snaps", torch.float32)
        if tuple(snaps.shape) != shape:
            raise ValueError("snaps must be %s" % (shape,))
    _check(lib().gdn_chunk_prefill_snapshots(
        _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S0), _ptr(a["o"]), _ptr(a["S_T"]),
        a["B"], a["T"], a["H"], a["dk"], a["dv"], chunk, _ptr(cu_seqlens), a["n_seqs"], a["io"], float(scale),
        int(snap_every), _ptr(snaps) if n_snap > 0 else None, _ptr(a["workspace"]), a["workspace"].numel(),
        _stream(q.device)))
    return a["o"], a["S_T"], snaps


def gdn_chunk_prefill_snapshots_ex(q, k, v, g, beta, S0=None, *, snap_every, flags=0, chunk=64, cu_seqlens=None,
                                   scale=1.0, o=None, S_T=None, snaps=None, store_state=True, workspace=None):
    """Snapshots with grouped key heads and input transforms; see ``gdn_chunk_prefill_snapshots_ex``.

    Shapes as ``gdn_chunk_prefill_grouped``; returns ``(o, S_T, snaps)`` as ``gdn_chunk_prefill_snapshots``.
    """
    a = _prefill_args(q, k, v, g, beta, S0, chunk, cu_seqlens, o, S_T, store_state, workspace, grouped=True)
    n_snap = max(0, (a["T"] - 1) // (int(snap_every) * chunk)) if snap_every >= 1 else 0
    shape = (a["n"], n_snap, a["H"], a["dv"], a["dk"])
    if snaps is None:
        snaps = torch.zeros(shape, device=q.device, dtype=torch.float32)
    else:
        _dev(snaps, "snaps", torch.float32)
        if tuple(snaps.shape) != shape:
            raise ValueError("snaps must be %s" % (shape,))
    _check(lib().gdn_chunk_prefill_snapshots_ex(
        _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S0), _ptr(a["o"]), _ptr(a["S_T"]),
        a["B"], a["T"], a["H"], a["HK"], a["dk"], a["dv"], chunk, _ptr(cu_seqlens), a["n_seqs"], a["io"],
        float(scale), int(flags), int(snap_every), _ptr(snaps) if n_snap > 0 else None, _ptr(a["workspace"]),
        a["workspace"].numel(), _stream(q.device)))
    return a["o"], a["S_T"], snaps


def gdn_decode_step(q, k, v, g, beta, S, *, scale=1.0, o=None):
    """One decode step; ``S`` [B,H,dv,dk] fp32 is updated in place.  Returns o [B,H,dv]."""
    return _decode(q, k, v, g, beta, S, scale, o, grouped=False)


def gdn_decode_step_grouped(q, k, v, g, beta, S, *, scale=1.0, o=None):
    """One decode step with grouped key heads: q, k [B,H_k,dk], v [B,H,dv]; ``S`` updated in place.  Returns o."""
    return _decode(q, k, v, g, beta, S, scale, o, grouped=True)


def gdn_decode_step_ex(q, k, v, g, beta, S, *, flags=0, scale=1.0, o=None):
    """One decode step with in-kernel input transforms (``flags`` as ``gdn_chunk_prefill_ex``).  Returns o."""
    return _decode(q, k, v, g, beta, S, scale, o, grouped=True, flags=flags)


def _decode(q, k, v, g, beta, S, scale, o, grouped, flags=None):
    if q.dtype not in _IO:
        raise TypeError("q must be float32 or bfloat16")
    io = _IO[q.dtype]
    for name, t in (("q", q), ("k", k), ("v", v)):
        _dev(t, name, q.dtype)
    _dev(g, "g", torch.float32)
    _dev(beta, "beta", torch.float32)
    _dev(S, "S", torch.float32)
    B, HK, dk = q.shape
    H = v.shape[1] if grouped else HK
    dv = v.shape[-1]
    if k.shape != q.shape or tuple(v.shape[:2]) != (B, H) or tuple(g.shape) != (B, H) \
            or beta.shape != g.shape or tuple(S.shape) != (B, H, dv, dk):
        raise ValueError("inconsistent decode shapes")
    if o is None:
        o = torch.empty_like(v)
    else:
        _dev(o, "o", q.dtype)
    if flags is not None:
        _check(lib().gdn_decode_step_ex(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S), _ptr(o),
                                        B, H, HK, dk, dv, io, float(scale), int(flags), _stream(q.device)))
    elif grouped:
        _check(lib().gdn_decode_step_grouped(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S), _ptr(o),
                                             B, H, HK, dk, dv, io, float(scale), _stream(q.device)))
    else:
        _check(lib().gdn_decode_step(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(S), _ptr(o),
                                     B, H, dk, dv, io, float(scale), _stream(q.device)))
    return o


def gdn_attention_prefill(q, k, v, *, scale=None, cu_seqlens=None, o=None):
    """Causal softmax attention; see ``gdn_attention_prefill`` in include/gdn.h.

    q [B,T,H,d] and k, v [B,T,H_kv,d] bf16 CUDA tensors; ``scale`` defaults to
    1/sqrt(d).  Packed sequences: B == 1 and ``cu_seqlens`` an int32 CUDA tensor
    [n+1].  Returns o [B,T,H,d] bf16.
    """
    n_seqs = 0
    if cu_seqlens is not None:
        _dev(cu_seqlens, "cu_seqlens", torch.int32)
        n_seqs = cu_seqlens.numel() - 1
    for name, t in (("q", q), ("k", k), ("v", v)):
        _dev(t, name, torch.bfloat16)
    B, T, H, d = q.shape
    Hkv = k.shape[2]
    if tuple(k.shape) != (B, T, Hkv, d) or v.shape != k.shape:
        raise ValueError("inconsistent shapes q%s k%s v%s" % (tuple(q.shape), tuple(k.shape), tuple(v.shape)))
    if o is None:
        o = torch.empty_like(q)
    else:
        _dev(o, "o", torch.bfloat16)
    sc = float(scale) if scale is not None else 1.0 / float(d) ** 0.5
    _check(lib().gdn_attention_prefill(_ptr(q), _ptr(k), _ptr(v), _ptr(o), B, T, H, Hkv, d, _ptr(cu_seqlens), n_seqs,
                                       GDN_BF16, sc, _stream(q.device)))
    return o
