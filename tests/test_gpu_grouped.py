"""GPU parity of grouped key heads (through the C ABI) against the fp64 oracle.

q and k carry H_k heads and value head h reads key head h // (H // H_k)
(``gdn_chunk_prefill_grouped``, ``gdn_decode_step_grouped``).  The oracle is
``oracle.recurrence_grouped``: the token-by-token definition with each value
head given its key head.  Bars as the other parity tests (max|x - ref| /
max|ref| per output tensor: 2e-4 fp32 io, 2e-2 bf16 io).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_14568_amd as gdn
from paper_2607_14568_amd import inputs

pytestmark = pytest.mark.gpu
TOL = {"f32": 2e-4, "bf16": 2e-2}
f64 = inputs.as_f64


def _dev(x):
    return {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in x.items()}


def _check(x, io, label, flags=None, segments=0):
    print("case:", label, flush=True)
    d = _dev(x)
    if flags is None:
        o, ST = gdn.gdn_chunk_prefill_grouped(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"],
                                              cu_seqlens=d["cu_seqlens"])
    else:
        o, ST = gdn.gdn_chunk_prefill_ex(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], flags=flags,
                                         segments=segments, cu_seqlens=d["cu_seqlens"])
    torch.cuda.synchronize()
    cu = None if x["cu_seqlens"] is None else x["cu_seqlens"].numpy()
    o_ref, ST_ref = oracle.recurrence_grouped(f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["g"]), f64(x["beta"]),
                                              f64(x["S0"]), cu_seqlens=cu)
    eo, es = oracle.max_rel_err(f64(o), o_ref), oracle.max_rel_err(f64(ST), ST_ref)
    print("  max rel err o=%.3e S_T=%.3e" % (eo, es), flush=True)
    assert np.isfinite(f64(o)).all() and np.isfinite(f64(ST)).all()
    assert eo < TOL[io], (label, eo)
    assert es < TOL[io], (label, es)
    return o, ST


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 128), (64, 128)])
@pytest.mark.parametrize("H,Hk", [(4, 2), (4, 1), (6, 3)])
@pytest.mark.parametrize("T", [65, 200])
def test_grouped_dense(io, dk, dv, H, Hk, T):
    x = inputs.make_prefill(B=2, T=T, H=H, H_k=Hk, dk=dk, dv=dv, io=io, seed=300 + T + H * 5 + Hk + dk + dv,
                            s0_std=0.05)
    _check(x, io, "grouped B=2 T=%d H=%d H_k=%d dk=%d dv=%d %s" % (T, H, Hk, dk, dv, io))


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_grouped_ragged(io):
    """Empty, one-token, whole-chunk and ragged-tail sequences packed together."""
    x = inputs.make_prefill(B=1, T=0, H=4, H_k=2, dk=128, dv=128, io=io, seed=311, s0_std=0.05,
                            lengths=[0, 1, 64, 130, 333])
    _check(x, io, "grouped ragged lengths 0,1,64,130,333 H=4 H_k=2 %s" % io)


def test_grouped_full_size_one_launch():
    """T=10240, 16 value heads over 8 key heads, bf16: the one-launch form at the timed shape."""
    x = inputs.make_prefill(B=1, T=10240, H=16, H_k=8, dk=128, dv=128, io="bf16", seed=1002, s0_std=0.02,
                            g_shift=2.0)
    _check(x, "bf16", "grouped T=10240 H=16 H_k=8 bf16")


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_grouped_segment_parallel(io):
    """The split form over two value heads sharing one key head (forced to 4 segments)."""
    x = inputs.make_prefill(B=1, T=64 * 40 + 9, H=2, H_k=1, dk=128, dv=128, io=io, seed=312, s0_std=0.05)
    _check(x, io, "grouped segments=4 T=%d H=2 H_k=1 %s" % (64 * 40 + 9, io), flags=gdn.GDN_PLAN_SEGMENTED, segments=4)


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_grouped_with_all_key_heads_is_the_plain_call(io):
    """H_k = H through the grouped entry point is gdn_chunk_prefill bit for bit."""
    x = _dev(inputs.make_prefill(B=2, T=150, H=3, dk=64, dv=128, io=io, seed=313, s0_std=0.05))
    a = gdn.gdn_chunk_prefill(x["q"], x["k"], x["v"], x["g"], x["beta"], x["S0"])
    b = gdn.gdn_chunk_prefill_grouped(x["q"], x["k"], x["v"], x["g"], x["beta"], x["S0"])
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(128, 128), (64, 128)])
def test_grouped_decode(io, dk, dv):
    print("case: grouped decode", io, dk, dv, flush=True)
    y = inputs.make_decode(B=6, H=8, H_k=2, dk=dk, dv=dv, io=io, seed=320 + dk + dv, pool=4)
    d = {k: v.cuda() for k, v in y.items()}
    S = d["S"].clone()
    S_ref = f64(y["S"])
    tol = TOL[io]
    for i in range(8):
        j = i % 4
        o = gdn.gdn_decode_step_grouped(d["q"][j], d["k"][j], d["v"][j], d["g"][j], d["beta"][j], S)
        o_ref, S_ref = oracle.decode_step_grouped(f64(y["q"][j]), f64(y["k"][j]), f64(y["v"][j]), f64(y["g"][j]),
                                                  f64(y["beta"][j]), S_ref)
        assert oracle.max_rel_err(f64(o), o_ref) < tol, i
    assert oracle.max_rel_err(f64(S), S_ref) < tol
