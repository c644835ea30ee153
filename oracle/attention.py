"""Causal softmax attention in fp64 -- TEST INFRASTRUCTURE ONLY (the parity oracle of
``gdn_attention_prefill``; only tests/, __graft_entry__.smoke() and bench.py's CPU
baseline use it).

The definition (section 5: scores Q K^T per head, a softmax over each query's causal
prefix, the product with V; grouped query heads share a key/value head), written out
per (sequence, head) with a library matrix product as the only building block:

    S = scale Q K^T,   S_ij = -inf for j > i,   P = rowwise softmax(S),   O = P V.
"""
from __future__ import annotations

import numpy as np


def causal_attention(q, k, v, scale, rows=None):
    """q [B,T,H,d]; k, v [B,T,H_kv,d] (H_kv divides H; head h reads key/value head h // (H // H_kv)).

    Returns o [B,T,H,d] in fp64, or only the query positions ``rows`` ([B,len(rows),H,d]).
    """
    q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
    B, T, H, d = q.shape
    Hkv = k.shape[2]
    assert k.shape == (B, T, Hkv, d) and v.shape == k.shape and H % Hkv == 0
    idx = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    o = np.zeros((B, len(idx), H, d))
    for b in range(B):
        for h in range(H):
            kh = h // (H // Hkv)
            s = scale * (q[b, idx, h] @ k[b, :, kh].T)             # [rows, T]
            s[np.arange(T)[None, :] > idx[:, None]] = -np.inf      # keys after the query
            s -= s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            o[b, :, h] = p @ v[b, :, kh]
    return o
