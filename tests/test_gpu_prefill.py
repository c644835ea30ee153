"""GPU parity of the chunked prefill (through the C ABI) against the fp64 oracle.

Metric: max|x - ref| / max|ref| per output tensor (o and S_T separately), and the same bar on every
(sequence, head) slice against that slice's largest value.  Bars: 2e-4 for fp32 io, 2e-2 for bf16
io (bf16 q, k, v, o with fp32 state).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_14568_amd as gdn
import parity
from paper_2607_14568_amd import inputs

pytestmark = pytest.mark.gpu
TOL = {"f32": 2e-4, "bf16": 2e-2}
f64 = inputs.as_f64


def _dev(x):
    return {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in x.items()}


def _run(x, **kw):
    d = _dev(x)
    o, ST = gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"],
                                  cu_seqlens=d["cu_seqlens"], **kw)
    torch.cuda.synchronize()
    return o, ST


def _ref(x, scale=1.0):
    cu = None if x["cu_seqlens"] is None else x["cu_seqlens"].numpy()
    return oracle.recurrence(f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["g"]), f64(x["beta"]),
                             f64(x["S0"]), cu_seqlens=cu, scale=scale)


def _check(x, io, label, scale=1.0):
    print("case:", label, flush=True)
    o, ST = _run(x, scale=scale)
    o_ref, ST_ref = _ref(x, scale)
    cu = None if x["cu_seqlens"] is None else x["cu_seqlens"].numpy()
    parity.check(f64(o), o_ref, f64(ST), ST_ref, TOL[io], label, cu_seqlens=cu)
    return o, ST


# ------------------------------------------------------------------ the named workloads
@pytest.mark.parametrize("name", ["tiny_f32", "prefill_2k_f32", "prefill_10k_bf16",
                                  "prefill_10k_bf16_slow", "ragged_8seq_bf16"])
def test_workload_parity(name):
    w = inputs.WORKLOADS[name]
    _check(inputs.make_workload(name), w.io, name)


# ------------------------------------------------------------------ sweeps
@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
@pytest.mark.parametrize("T", [1, 5, 63, 64, 65, 200])
def test_shapes_and_tails(io, dk, dv, T):
    x = inputs.make_prefill(B=2, T=T, H=3, dk=dk, dv=dv, io=io, seed=T * 7 + dk + dv, s0_std=0.1)
    _check(x, io, "B=2 T=%d H=3 dk=%d dv=%d %s" % (T, dk, dv, io))


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_no_initial_state_and_scale(io):
    x = inputs.make_prefill(B=1, T=130, H=2, dk=128, dv=128, io=io, seed=3)
    assert x["S0"] is None
    _check(x, io, "S0=None scale=0.088", scale=128 ** -0.5)


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("case", ["alpha0", "alpha1", "beta0", "beta1", "mixed_extreme"])
def test_extreme_gates(io, case):
    x = inputs.make_prefill(B=1, T=150, H=2, dk=128, dv=64, io=io, seed=11, s0_std=0.1)
    g, b = x["g"], x["beta"]
    if case == "alpha0":
        g.fill_(-1e4)                   # alpha underflows: no memory across tokens
    elif case == "alpha1":
        g.zero_()                       # plain delta rule
    elif case == "beta0":
        b.zero_()                       # pure decay of S0; milder decay keeps
        g.mul_(0.05)                    # exp(sum g) S0 inside the fp32 range
    elif case == "beta1":
        b.fill_(1.0)
    else:
        g[:, ::3] = -1e4
        g[:, 1::3] = 0.0
        b[:, ::2] = 1.0
        b[:, 1::4] = 0.0
    _check(x, io, "gates %s %s" % (case, io))


def test_ragged_edge_lengths():
    lens = [0, 1, 63, 64, 65, 0, 130, 7]
    x = inputs.make_prefill(B=1, T=0, H=2, dk=128, dv=128, io="bf16", seed=5, s0_std=0.05, lengths=lens)
    o, ST = _check(x, "bf16", "ragged lens=%s" % lens)
    # empty sequences keep their initial state exactly
    for s, n in enumerate(lens):
        if n == 0:
            assert torch.equal(ST[s].cpu(), x["S0"][s])


def test_empty_prompt_returns_initial_state():
    x = inputs.make_prefill(B=2, T=0, H=2, dk=64, dv=64, io="f32", seed=1, s0_std=0.1)
    o, ST = _run(x)
    assert o.numel() == 0
    assert torch.equal(ST.cpu(), x["S0"])
    x["S0"] = None
    o, ST = _run(x)
    assert torch.count_nonzero(ST) == 0


# ------------------------------------------------------------------ invariants of the GPU path
def test_state_passing_two_calls_equal_one():
    x = inputs.make_prefill(B=1, T=300, H=4, dk=128, dv=128, io="f32", seed=21, s0_std=0.05)
    o, ST = _run(x)
    a = {k: (v[:, :128] if k in ("q", "k", "v", "g", "beta") else v) for k, v in x.items()}
    b = {k: (v[:, 128:].contiguous() if k in ("q", "k", "v", "g", "beta") else v) for k, v in x.items()}
    oa, Sa = _run(a)
    b["S0"] = Sa.cpu()
    ob, Sb = _run(b)
    assert oracle.max_rel_err(f64(torch.cat([oa, ob], 1)), f64(o)) < 1e-5
    assert oracle.max_rel_err(f64(Sb), f64(ST)) < 1e-5


def test_ragged_equals_separate_calls():
    lens = [100, 37, 256]
    x = inputs.make_prefill(B=1, T=0, H=2, dk=128, dv=128, io="bf16", seed=23, s0_std=0.05, lengths=lens)
    o, ST = _run(x)
    cu = x["cu_seqlens"].tolist()
    for s in range(len(lens)):
        sl = slice(cu[s], cu[s + 1])
        y = {k: (v[:, sl].contiguous() if k in ("q", "k", "v", "g", "beta") else v) for k, v in x.items()}
        y["S0"] = x["S0"][s:s + 1]
        y["cu_seqlens"] = None
        os_, Ss = _run(y)
        assert torch.equal(os_, o[:, sl]), s          # same kernels, same chunk grid: bitwise
        assert torch.equal(Ss[0], ST[s]), s


def test_prefill_T1_matches_decode_step():
    x = inputs.make_prefill(B=3, T=1, H=4, dk=128, dv=128, io="f32", seed=29, s0_std=0.05)
    o, ST = _run(x)
    d = _dev(x)
    S = d["S0"].clone()
    od = gdn.gdn_decode_step(d["q"][:, 0].contiguous(), d["k"][:, 0].contiguous(), d["v"][:, 0].contiguous(),
                             d["g"][:, 0].contiguous(), d["beta"][:, 0].contiguous(), S)
    torch.cuda.synchronize()
    assert oracle.max_rel_err(f64(od), f64(o[:, 0])) < 1e-5
    assert oracle.max_rel_err(f64(S), f64(ST)) < 1e-5


def test_bitwise_deterministic_and_every_output_written():
    x = inputs.make_prefill(B=1, T=333, H=4, dk=128, dv=128, io="bf16", seed=31, s0_std=0.05)
    d = _dev(x)
    outs = []
    for _ in range(2):
        o = torch.full_like(d["v"], float("nan"))
        ST = torch.full_like(d["S0"], float("nan"))
        gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], o=o, S_T=ST)
        torch.cuda.synchronize()
        assert torch.isfinite(o).all() and torch.isfinite(ST).all()
        outs.append((o.clone(), ST.clone()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


def test_in_place_state():
    x = inputs.make_prefill(B=2, T=100, H=2, dk=64, dv=128, io="f32", seed=37, s0_std=0.05)
    o_ref, ST_ref = _ref(x)
    d = _dev(x)
    S = d["S0"].clone()
    o, ST = gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], S, S_T=S)
    torch.cuda.synchronize()
    assert ST.data_ptr() == S.data_ptr()
    assert oracle.max_rel_err(f64(S), ST_ref) < 2e-4
    assert oracle.max_rel_err(f64(o), o_ref) < 2e-4


def test_workspace_contents_do_not_matter():
    x = inputs.make_prefill(B=1, T=200, H=2, dk=128, dv=128, io="bf16", seed=41, s0_std=0.05)
    d = _dev(x)
    need = gdn.gdn_chunk_prefill_workspace_bytes(1, 200, 2, 128, 128, 64, 0, gdn.GDN_BF16)
    ws = torch.full((need,), 0xFF, dtype=torch.uint8, device="cuda")
    o1, S1 = gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], workspace=ws)
    ws.fill_(0)
    o2, S2 = gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(S1, S2)


def test_invalid_ragged_offsets_are_clamped_not_faulting():
    """Offsets outside the contract are clamped on the device into a partition of [0, T]."""
    x = inputs.make_prefill(B=1, T=200, H=2, dk=64, dv=64, io="f32", seed=43, s0_std=0.05)
    d = _dev(x)
    cu = torch.tensor([0, 150, 90, 500], dtype=torch.int32, device="cuda")   # decreasing, beyond T
    o, ST = gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"],
                                  torch.zeros(3, 2, 64, 64, device="cuda"), cu_seqlens=cu)
    torch.cuda.synchronize()
    # clamped partition: [0,150), [150,150), [150,200)
    ref_o, ref_S = oracle.recurrence(f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["g"]), f64(x["beta"]),
                                     None, cu_seqlens=[0, 150, 150, 200])
    assert oracle.max_rel_err(f64(o), ref_o) < 2e-4
    assert oracle.max_rel_err(f64(ST), ref_S) < 2e-4


def test_workspace_reused_across_calls_with_different_inputs():
    """One workspace, three calls with different inputs and shapes: no call may read another call's chunk matrices."""
    need = max(gdn.gdn_chunk_prefill_workspace_bytes(1, T, 4, 128, 128, 64, 0, gdn.GDN_BF16) for T in (300, 200))
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    for i, (T, seed) in enumerate([(300, 51), (300, 52), (200, 53)]):
        x = inputs.make_prefill(B=1, T=T, H=4, dk=128, dv=128, io="bf16", seed=seed, s0_std=0.05)
        print("case: call %d T=%d seed=%d" % (i, T, seed), flush=True)
        d = _dev(x)
        o, ST = gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], workspace=ws)
        torch.cuda.synchronize()
        o_ref, ST_ref = _ref(x)
        assert oracle.max_rel_err(f64(o), o_ref) < TOL["bf16"], i
        assert oracle.max_rel_err(f64(ST), ST_ref) < TOL["bf16"], i


@pytest.mark.parametrize("T", [200, 700])
def test_dense_batch_through_two_launches(T):
    """B=2, H=16, dv=128 gives 256 chain workgroups: no CUs are left beside the
    chain, so the chunk terms run as their own launch before it."""
    x = inputs.make_prefill(B=2, T=T, H=16, dk=128, dv=128, io="bf16", seed=T + 5, s0_std=0.05)
    _check(x, "bf16", "B=2 T=%d H=16 bf16 (two launches)" % T)


@pytest.mark.parametrize("B,H,T", [(1, 8, 700), (2, 8, 600), (1, 24, 450)])
def test_one_launch_item_order_per_xcd(B, H, T):
    """One launch with 8 | H (chunk-terms items walked per XCD, several sequences and heads per
    workgroup) and with the poller observing flags ahead of the loaders through the tail chunks."""
    x = inputs.make_prefill(B=B, T=T, H=H, dk=128, dv=128, io="bf16", seed=B * 100 + H + T, s0_std=0.05)
    _check(x, "bf16", "B=%d T=%d H=%d bf16 (one launch, per-XCD item order)" % (B, T, H))
