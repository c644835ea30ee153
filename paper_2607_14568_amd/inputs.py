"""Seeded synthetic inputs for the gated delta-rule path.

This module only draws random numbers and shapes them into the input
distributions of the workloads; it holds none of the method's arithmetic.
Both the parity oracle and the HIP path consume what it returns.

Recipe (paper, section 2.2: 16 value heads, H_k = H_v = 128; section 5: a
10k-token long-context tier):
  * ``numpy.random.default_rng(seed)``; draw order: (ragged lengths,) q, k, v,
    beta logits, decay logits, initial state.
  * q, k ~ N(0,1), L2-normalised over the head dimension in fp64, then rounded
    to the io dtype (bf16 with round-to-nearest-even, or fp32);
  * v ~ N(0,1) rounded to the io dtype;
  * beta = sigmoid(N(0,1)) in fp32;
  * g = -softplus(N(0,1) + shift) in fp32 (alpha = exp(g));
  * S0 = std * N(0,1) in fp32, or absent.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

IO_DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclass
class Workload:
    name: str
    B: int
    T: int
    H: int
    dk: int
    dv: int
    io: str                      # "f32" | "bf16"
    seed: int
    s0_std: float = 0.0          # 0 -> no initial state
    g_shift: float = 0.0
    ragged: int = 0              # number of packed sequences (0 -> dense)
    len_range: tuple = (512, 4096)
    decode: bool = False
    pool: int = 16               # decode: distinct tokens cycled over steps
    chunk: int = 64
    notes: str = field(default="")


WORKLOADS = {
    # tiny fp32 case the oracle finishes instantly
    "tiny_f32": Workload("tiny_f32", B=1, T=256, H=2, dk=64, dv=64, io="f32", seed=1000),
    # backbone-shaped prefill, 2k context, carried state
    "prefill_2k_f32": Workload("prefill_2k_f32", B=1, T=2048, H=16, dk=128, dv=128, io="f32",
                               seed=1001, s0_std=0.02),
    # long-context prefill: 10240 tokens, bf16 io, fp32 state (the timed workload)
    "prefill_10k_bf16": Workload("prefill_10k_bf16", B=1, T=10240, H=16, dk=128, dv=128,
                                 io="bf16", seed=1002, s0_std=0.02, g_shift=2.0),
    # same shape with slow decay (mean alpha ~ 0.84): long-memory numerics
    "prefill_10k_bf16_slow": Workload("prefill_10k_bf16_slow", B=1, T=10240, H=16, dk=128,
                                      dv=128, io="bf16", seed=1012, s0_std=0.02, g_shift=-2.0),
    # one device's share of the 16 heads under an 8-way head split: the sequential chain
    # leaves most CUs idle, so the prefill takes the segment-parallel form
    "prefill_10k_h2_bf16": Workload("prefill_10k_h2_bf16", B=1, T=10240, H=2, dk=128, dv=128,
                                    io="bf16", seed=1005, s0_std=0.02, g_shift=2.0),
    "prefill_10k_h2_f32": Workload("prefill_10k_h2_f32", B=1, T=10240, H=2, dk=128, dv=128,
                                   io="f32", seed=1006, s0_std=0.02, g_shift=2.0),
    # 8 packed sequences of uniform length in [512, 4096], per-sequence state
    "ragged_8seq_bf16": Workload("ragged_8seq_bf16", B=1, T=0, H=16, dk=128, dv=128, io="bf16",
                                 seed=1003, s0_std=0.02, ragged=8),
    # decode: 64 sequences, one token each per step, resident fp32 state
    "decode_b64_f32": Workload("decode_b64_f32", B=64, T=1, H=16, dk=128, dv=128, io="f32",
                               seed=1004, s0_std=0.02, decode=True),
    # the same step over 512 sequences: 537 MB of state, larger than the 256 MB Infinity Cache
    "decode_b512_f32": Workload("decode_b512_f32", B=512, T=1, H=16, dk=128, dv=128, io="f32",
                                seed=1014, s0_std=0.02, decode=True, pool=4),
}


def _round_io(x64: np.ndarray, io: str) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x64, dtype=np.float64)).to(IO_DTYPES[io])


def _l2n(x: np.ndarray) -> np.ndarray:
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def make_prefill(B, T, H, dk, dv, io="f32", seed=0, s0_std=0.0, g_shift=0.0,
                 lengths=None, ragged=0, len_range=(512, 4096), H_k=None, raw=False):
    """Dense (B,T) or ragged (``ragged`` sequences, or explicit ``lengths``) inputs.

    Returns a dict of CPU torch tensors: q,k [B,T,H_k,dk] (H_k = H unless given)
    and v [B,T,H,dv] in the io dtype; g, beta [B,T,H] fp32; S0 [n_seq,H,dv,dk]
    fp32 or None; cu_seqlens int32 [n_seq+1] or None.  ``raw``: the same draws
    before the recipe's last steps -- q, k not scaled to unit length, and g, beta
    holding the logits a = N(0,1) + g_shift, b = N(0,1) (for the entry points that
    take GDN_QK_L2NORM and GDN_GATE_LOGITS).
    """
    H_k = H if H_k is None else H_k
    rng = np.random.default_rng(seed)
    cu = None
    if ragged or lengths is not None:
        if lengths is None:
            lengths = rng.integers(len_range[0], len_range[1] + 1, size=ragged)
        lengths = np.asarray(lengths, dtype=np.int64)
        cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
        B, T = 1, int(cu[-1])
        n_seq = len(lengths)
    else:
        n_seq = B
    q = rng.standard_normal((B, T, H_k, dk))
    k = rng.standard_normal((B, T, H_k, dk))
    v = rng.standard_normal((B, T, H, dv))
    b_logit = rng.standard_normal((B, T, H))
    a_logit = rng.standard_normal((B, T, H)) + g_shift
    if raw:
        beta, g = b_logit, a_logit
    else:
        q, k = _l2n(q), _l2n(k)
        beta = 1.0 / (1.0 + np.exp(-b_logit))
        g = -np.logaddexp(0.0, a_logit)
    S0 = s0_std * rng.standard_normal((n_seq, H, dv, dk)) if s0_std > 0 else None
    return dict(
        q=_round_io(q, io), k=_round_io(k, io), v=_round_io(v, io),
        g=torch.from_numpy(g.astype(np.float32)),
        beta=torch.from_numpy(beta.astype(np.float32)),
        S0=None if S0 is None else torch.from_numpy(S0.astype(np.float32)),
        cu_seqlens=None if cu is None else torch.from_numpy(cu),
    )


def make_decode(B, H, dk, dv, io="f32", seed=0, s0_std=0.02, pool=16, H_k=None, raw=False):
    """Decode inputs: a pool of ``pool`` tokens per sequence, cycled by step index.

    Returns q,k [pool,B,H_k,dk] (H_k = H unless given), v [pool,B,H,dv] (io
    dtype); g, beta [pool,B,H] fp32; S [B,H,dv,dk] fp32.  ``raw`` as make_prefill.
    """
    H_k = H if H_k is None else H_k
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((pool, B, H_k, dk))
    k = rng.standard_normal((pool, B, H_k, dk))
    v = rng.standard_normal((pool, B, H, dv))
    b_logit = rng.standard_normal((pool, B, H))
    a_logit = rng.standard_normal((pool, B, H))
    if raw:
        beta, g = b_logit, a_logit
    else:
        q, k = _l2n(q), _l2n(k)
        beta = 1.0 / (1.0 + np.exp(-b_logit))
        g = -np.logaddexp(0.0, a_logit)
    S = s0_std * rng.standard_normal((B, H, dv, dk))
    return dict(q=_round_io(q, io), k=_round_io(k, io), v=_round_io(v, io),
                g=torch.from_numpy(g.astype(np.float32)),
                beta=torch.from_numpy(beta.astype(np.float32)),
                S=torch.from_numpy(S.astype(np.float32)))


def make_attention(B, T, H, H_kv, d, seed=0):
    """Attention inputs: q [B,T,H,d], k and v [B,T,H_kv,d], entries N(0,1), bf16."""
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, T, H, d), dtype=np.float32)
    k = rng.standard_normal((B, T, H_kv, d), dtype=np.float32)
    v = rng.standard_normal((B, T, H_kv, d), dtype=np.float32)
    return dict(q=torch.from_numpy(q).to(torch.bfloat16), k=torch.from_numpy(k).to(torch.bfloat16),
                v=torch.from_numpy(v).to(torch.bfloat16))


def make_workload(name: str):
    w = WORKLOADS[name]
    if w.decode:
        return make_decode(w.B, w.H, w.dk, w.dv, w.io, w.seed, w.s0_std, w.pool)
    return make_prefill(w.B, w.T, w.H, w.dk, w.dv, w.io, w.seed, w.s0_std, w.g_shift,
                        ragged=w.ragged, len_range=w.len_range)


def as_f64(t):
    """Exact fp64 copy of a CPU/GPU tensor's values (None passes through)."""
    if t is None:
        return None
    return t.detach().to("cpu", torch.float64).numpy()
