"""GPU parity of the in-kernel input transforms (gdn_chunk_prefill_ex, gdn_decode_step_ex).

GDN_QK_L2NORM: q and k arrive unnormalised and every row is used as
x / sqrt(|x|^2 + 1e-6); GDN_GATE_LOGITS: g and beta arrive as logits, g =
-softplus(a), beta = sigmoid(b).  The oracle (``oracle.recurrence_ex``) applies
the same transforms in fp64 and runs the token-by-token definition.  Bars as
the other parity tests (max|x - ref| / max|ref|: 2e-4 fp32 io, 2e-2 bf16 io).
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
L2, GATES = gdn.GDN_QK_L2NORM, gdn.GDN_GATE_LOGITS


def _dev(x):
    return {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in x.items()}


def _check(x, io, flags, label, segments=0):
    print("case:", label, "flags=%d" % flags, flush=True)
    d = _dev(x)
    o, ST = gdn.gdn_chunk_prefill_ex(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], flags=flags,
                                     segments=segments, cu_seqlens=d["cu_seqlens"])
    torch.cuda.synchronize()
    cu = None if x["cu_seqlens"] is None else x["cu_seqlens"].numpy()
    o_ref, ST_ref = oracle.recurrence_ex(f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["g"]), f64(x["beta"]),
                                         f64(x["S0"]), cu_seqlens=cu, qk_l2norm=bool(flags & L2),
                                         gate_logits=bool(flags & GATES))
    eo, es = oracle.max_rel_err(f64(o), o_ref), oracle.max_rel_err(f64(ST), ST_ref)
    print("  max rel err o=%.3e S_T=%.3e" % (eo, es), flush=True)
    assert np.isfinite(f64(o)).all() and np.isfinite(f64(ST)).all()
    assert eo < TOL[io], (label, eo)
    assert es < TOL[io], (label, es)
    return o, ST


def _raw(flags, **kw):
    """Inputs with q, k unnormalised when L2 is asked for, and logits for g, beta when GATES is."""
    x = inputs.make_prefill(raw=True, **kw)
    ref = inputs.make_prefill(raw=False, **kw)   # the same draws with the recipe's transforms
    if not flags & L2:
        x["q"], x["k"] = ref["q"], ref["k"]
    if not flags & GATES:
        x["g"], x["beta"] = ref["g"], ref["beta"]
    return x


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("flags", [L2, GATES, L2 | GATES])
@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 128), (128, 64)])
@pytest.mark.parametrize("T", [65, 200])
def test_preops_dense(io, flags, dk, dv, T):
    x = _raw(flags, B=2, T=T, H=4, H_k=2, dk=dk, dv=dv, io=io, seed=400 + T + dk + dv + flags, s0_std=0.05)
    _check(x, io, flags, "ex B=2 T=%d H=4 H_k=2 dk=%d dv=%d %s" % (T, dk, dv, io))


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_preops_ragged(io):
    x = _raw(L2 | GATES, B=1, T=0, H=4, dk=128, dv=128, io=io, seed=411, s0_std=0.05, lengths=[0, 1, 64, 130, 333])
    _check(x, io, L2 | GATES, "ex ragged lengths 0,1,64,130,333 %s" % io)


def test_preops_full_size_one_launch():
    """T=10240, H=16, bf16 from raw q, k and gate logits: the one-launch form with the transforms."""
    x = _raw(L2 | GATES, B=1, T=10240, H=16, dk=128, dv=128, io="bf16", seed=1002, s0_std=0.02, g_shift=2.0)
    _check(x, "bf16", L2 | GATES, "ex T=10240 H=16 bf16")


def test_preops_two_launches():
    """32 heads x 2 sequences fill the device with chain workgroups: chunk terms and chain as two launches."""
    x = _raw(L2 | GATES, B=2, T=300, H=32, dk=128, dv=128, io="bf16", seed=412, s0_std=0.05)
    _check(x, "bf16", L2 | GATES, "ex B=2 T=300 H=32 bf16")


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_preops_segment_parallel(io):
    x = _raw(L2 | GATES, B=1, T=64 * 30 + 5, H=2, dk=128, dv=128, io=io, seed=413, s0_std=0.05)
    _check(x, io, L2 | GATES | gdn.GDN_PLAN_SEGMENTED, "ex segments=4 T=%d H=2 %s" % (64 * 30 + 5, io), segments=4)


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_preops_zero_flags_is_the_grouped_call(io):
    x = _dev(inputs.make_prefill(B=2, T=150, H=4, H_k=2, dk=64, dv=128, io=io, seed=414, s0_std=0.05))
    a = gdn.gdn_chunk_prefill_grouped(x["q"], x["k"], x["v"], x["g"], x["beta"], x["S0"])
    b = gdn.gdn_chunk_prefill_ex(x["q"], x["k"], x["v"], x["g"], x["beta"], x["S0"], flags=0)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_preops_zero_key_rows(io):
    """Tokens whose key row is all zeros write nothing (their transformed key stays zero)."""
    x = _raw(L2 | GATES, B=1, T=130, H=2, dk=128, dv=128, io=io, seed=415, s0_std=0.05)
    x["k"][0, [0, 63, 64, 129]] = 0
    _check(x, io, L2 | GATES, "ex zero key rows %s" % io)


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(128, 128), (64, 128)])
def test_preops_decode(io, dk, dv):
    print("case: ex decode", io, dk, dv, flush=True)
    y = inputs.make_decode(B=6, H=4, H_k=2, dk=dk, dv=dv, io=io, seed=420 + dk + dv, pool=4, raw=True)
    d = {k: v.cuda() for k, v in y.items()}
    S = d["S"].clone()
    S_ref = f64(y["S"])
    for i in range(8):
        j = i % 4
        o = gdn.gdn_decode_step_ex(d["q"][j], d["k"][j], d["v"][j], d["g"][j], d["beta"][j], S, flags=L2 | GATES,
                                   scale=0.7)
        o_ref, S_ref = oracle.decode_step_ex(f64(y["q"][j]), f64(y["k"][j]), f64(y["v"][j]), f64(y["g"][j]),
                                             f64(y["beta"][j]), S_ref, qk_l2norm=True, gate_logits=True, scale=0.7)
        assert oracle.max_rel_err(f64(o), o_ref) < TOL[io], i
    assert oracle.max_rel_err(f64(S), S_ref) < TOL[io]
