"""GPU parity at sizes well past the timed workload (through the C ABI), against the fp64 oracle.

Long prompts, many packed sequences, many heads and a dense batch exercise the
index arithmetic of every kernel (sequence tables, chunk slots, 32-bit
in-chunk offsets over 64-bit bases) at scale.  The oracle still finishes each
case in seconds, so every output is compared.  Bars as the other parity tests.
"""
import pytest
import torch

import oracle
import paper_2607_14568_amd as gdn
import parity
from paper_2607_14568_amd import inputs

pytestmark = pytest.mark.gpu
TOL = {"f32": 2e-4, "bf16": 2e-2}
f64 = inputs.as_f64


def _check(x, io, label):
    print("case:", label, flush=True)
    d = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in x.items()}
    o, ST = gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], cu_seqlens=d["cu_seqlens"])
    torch.cuda.synchronize()
    del d
    cu = None if x["cu_seqlens"] is None else x["cu_seqlens"].numpy()
    o_ref, ST_ref = oracle.recurrence(f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["g"]), f64(x["beta"]),
                                      f64(x["S0"]), cu_seqlens=cu)
    parity.check(f64(o), o_ref, f64(ST), ST_ref, TOL[io], label, cu_seqlens=cu)


def test_long_prompt_32k_one_launch():
    """T = 32768 (512 chunks per head), 16 heads, bf16, slow decay: the one-launch form over a long chain."""
    x = inputs.make_prefill(B=1, T=32768, H=16, dk=128, dv=128, io="bf16", seed=500, s0_std=0.02, g_shift=-2.0)
    _check(x, "bf16", "T=32768 H=16 bf16 slow decay")


def test_many_packed_sequences():
    """48 sequences of 1..1200 tokens (chain workgroups in several rounds), bf16."""
    x = inputs.make_prefill(B=1, T=0, H=16, dk=128, dv=128, io="bf16", seed=501, s0_std=0.02, ragged=48,
                            len_range=(1, 1200))
    _check(x, "bf16", "ragged 48 sequences H=16 bf16")


def test_many_heads_f32():
    x = inputs.make_prefill(B=1, T=2048, H=64, dk=128, dv=128, io="f32", seed=502, s0_std=0.02)
    _check(x, "f32", "T=2048 H=64 f32")


def test_dense_batch_bf16():
    """8 sequences of 4096 tokens x 8 heads: 512 chain workgroups, two launches."""
    x = inputs.make_prefill(B=8, T=4096, H=8, dk=128, dv=64, io="bf16", seed=503, s0_std=0.02)
    _check(x, "bf16", "B=8 T=4096 H=8 dk=128 dv=64 bf16")
