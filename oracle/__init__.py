"""Parity oracle for the gated delta-rule path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library in
``paper_2607_14568_amd``) never imports it and shares no code with it.

Two independent CPU implementations live here, both in fp64:

* :func:`recurrence` -- the plain definition (paper, section 2.2 and section
  3.2): the token-by-token gated delta rule, in C (``gdn_oracle.c``), OpenMP
  over independent state rows.  This is THE parity oracle.
* :mod:`oracle.chunked` -- the intra-/inter-chunk form described in section
  3.2, in numpy, step by step.  It is pinned against :func:`recurrence` at
  every chunk size and is used to inspect the intermediate quantities the GPU
  path follows (never to produce expected values for the GPU).

Inputs are numpy arrays holding the exact values the GPU receives (bf16 or
fp32 values upcast to fp64 by the caller).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "gdn_oracle.c")
_lib = None


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (no fast-math: sums keep source order)."""
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(_SRC):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-Wall",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _SO)
    return _SO


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        lib = ctypes.CDLL(_SO)
        P = ctypes.c_void_p
        lib.oracle_gdn_recurrence.argtypes = [P, P, P, P, P, P, P, P, P, P, ctypes.c_int,
                                              ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                              ctypes.c_double, ctypes.c_int]
        lib.oracle_gdn_recurrence.restype = ctypes.c_int
        lib.oracle_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def recurrence(q, k, v, g, beta, S0=None, *, cu_seqlens=None, scale=1.0, n_threads=0,
               return_state=True):
    """Token-by-token gated delta rule in fp64 (section 2.2 / section 3.2).

    Dense:  q,k [B,T,H,dk]; v [B,T,H,dv]; g,beta [B,T,H]; S0 [B,H,dv,dk] or None.
    Ragged: B == 1 and ``cu_seqlens`` int array [N+1]; S0 [N,H,dv,dk] or None.
    Returns ``(o [B,T,H,dv], S_T [n_seq,H,dv,dk])`` in fp64.
    """
    q, k, v, g, beta = (_f64(x) for x in (q, k, v, g, beta))
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    assert k.shape == q.shape and v.shape[:3] == (B, T, H) and g.shape == (B, T, H)
    assert beta.shape == g.shape
    if cu_seqlens is None:
        starts = np.arange(B, dtype=np.int64) * T
        lens = np.full(B, T, dtype=np.int64)
    else:
        assert B == 1
        cu = np.asarray(cu_seqlens, dtype=np.int64)
        starts = np.ascontiguousarray(cu[:-1])
        lens = np.ascontiguousarray(cu[1:] - cu[:-1])
        assert (lens >= 0).all() and cu[0] == 0 and cu[-1] == T
    n_seq = len(starts)
    S0c = None if S0 is None else _f64(S0)
    if S0c is not None:
        assert S0c.shape == (n_seq, H, dv, dk)
    o = np.zeros((B, T, H, dv), dtype=np.float64)
    ST = np.zeros((n_seq, H, dv, dk), dtype=np.float64)
    rc = _load().oracle_gdn_recurrence(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                                       _ptr(S0c), _ptr(o), _ptr(ST),
                                       _ptr(starts), _ptr(lens), n_seq, H, dk, dv,
                                       float(scale), int(n_threads))
    if rc != 0:
        raise ValueError("oracle_gdn_recurrence rejected its arguments (code %d)" % rc)
    return (o, ST) if return_state else o


def expand_key_heads(x, H):
    """Query or key heads [..., H_k, d] -> one per value head [..., H, d].

    Grouped key heads (section 2.2 keeps one state per value head): value head h
    reads key head h // (H // H_k), so consecutive groups of H // H_k value heads
    share a query and key head.
    """
    x = _f64(x)
    Hk = x.shape[-2]
    assert H % Hk == 0, (H, Hk)
    return np.ascontiguousarray(x[..., np.arange(H) // (H // Hk), :])


def recurrence_grouped(q, k, v, g, beta, S0=None, **kw):
    """:func:`recurrence` with q,k [B,T,H_k,dk] shared by groups of value heads (v [B,T,H,dv])."""
    H = np.shape(v)[2]
    return recurrence(expand_key_heads(q, H), expand_key_heads(k, H), v, g, beta, S0, **kw)


def decode_step_grouped(q, k, v, g, beta, S, **kw):
    """:func:`decode_step` with q,k [B,H_k,dk] shared by groups of value heads (v [B,H,dv])."""
    H = np.shape(v)[1]
    return decode_step(expand_key_heads(q, H), expand_key_heads(k, H), v, g, beta, S, **kw)


L2_EPS = 1e-6   # of the unit-length transform of q and k


def l2_rows(x):
    """Each row (last axis) scaled to x / sqrt(|x|^2 + 1e-6): the kernels' GDN_QK_L2NORM transform."""
    x = _f64(x)
    return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + L2_EPS)


def gates_from_logits(a, b):
    """GDN_GATE_LOGITS: log-decay g = -softplus(a) = -log(1 + exp(a)), write strength beta = sigmoid(b)."""
    a, b = _f64(a), _f64(b)
    return -np.logaddexp(0.0, a), 1.0 / (1.0 + np.exp(-b))


def recurrence_ex(q, k, v, g, beta, S0=None, *, qk_l2norm=False, gate_logits=False, **kw):
    """:func:`recurrence_grouped` after the input transforms the _ex entry points apply in their kernels."""
    if qk_l2norm:
        q, k = l2_rows(q), l2_rows(k)
    if gate_logits:
        g, beta = gates_from_logits(g, beta)
    return recurrence_grouped(q, k, v, g, beta, S0, **kw)


def decode_step_ex(q, k, v, g, beta, S, *, qk_l2norm=False, gate_logits=False, **kw):
    """:func:`decode_step_grouped` after the same input transforms."""
    if qk_l2norm:
        q, k = l2_rows(q), l2_rows(k)
    if gate_logits:
        g, beta = gates_from_logits(g, beta)
    return decode_step_grouped(q, k, v, g, beta, S, **kw)


def decode_step(q, k, v, g, beta, S, *, scale=1.0, n_threads=0):
    """One token per sequence: q,k [B,H,dk]; v [B,H,dv]; g,beta [B,H]; S [B,H,dv,dk].

    It is the recurrence at T = 1 with the state passed in; returns (o, S_new).
    """
    q, k, v, g, beta = (_f64(x)[:, None] for x in (q, k, v, g, beta))
    o, S_new = recurrence(q, k, v, g, beta, S, scale=scale, n_threads=n_threads)
    return o[:, 0], S_new


def max_rel_err(x, ref) -> float:
    """max|x - ref| / max|ref| over one output tensor: the parity metric, the reading taken of
    the relative error section 3.2 quotes without a definition.  When ref is all zeros it is the
    absolute error max|x - ref|; empty tensors give 0.  x and ref must have the same shape."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if x.shape != ref.shape:
        raise ValueError("max_rel_err: shapes differ %s vs %s" % (x.shape, ref.shape))
    if ref.size == 0:
        return 0.0
    den = float(np.max(np.abs(ref)))
    num = float(np.max(np.abs(x - ref)))
    if den == 0.0:
        return num
    return num / den


def max_rel_err_slices(x, ref, index) -> float:
    """The largest :func:`max_rel_err` over the slices ``x[i], ref[i]`` for i in ``index`` (each
    slice against its own largest reference value); empty slices are skipped."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if x.shape != ref.shape:
        raise ValueError("max_rel_err_slices: shapes differ %s vs %s" % (x.shape, ref.shape))
    worst = 0.0
    for i in index:
        if ref[i].size:
            worst = max(worst, max_rel_err(x[i], ref[i]))
    return worst


def p99_rel_err(x, ref) -> float:
    """99th percentile over elements of |x - ref| / (|ref| + 1e-3 rms(ref)): reported beside the
    parity metric for information (it is not a bar)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if x.shape != ref.shape:
        raise ValueError("p99_rel_err: shapes differ %s vs %s" % (x.shape, ref.shape))
    if ref.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(ref * ref)))
    return float(np.percentile(np.abs(x - ref) / (np.abs(ref) + 1e-3 * rms), 99))
