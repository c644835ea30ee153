"""GPU parity of the state snapshots (gdn_chunk_prefill_snapshots) against the fp64 oracle.

Snapshot j of a sequence is its state after its first j * snap_every * 64 tokens;
the oracle's final state of that prefix is the reference.  Bars as for S_T:
max|x - ref| / max|ref| < 2e-4 (fp32 io), 2e-2 (bf16 io).
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
TOKEN = ("q", "k", "v", "g", "beta")


def _dev(x):
    return {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in x.items()}


def _prefix_state(x, s, t, scale=1.0):
    """Oracle state of sequence s after its first t tokens (dense input)."""
    S0 = None if x["S0"] is None else f64(x["S0"][s:s + 1])
    _, S = oracle.recurrence(*(f64(x[k][s:s + 1, :t]) for k in TOKEN), S0, scale=scale)
    return S[0]


def _snap(x, E, **kw):
    d = _dev(x)
    o, ST, sn = gdn.gdn_chunk_prefill_snapshots(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], snap_every=E,
                                                cu_seqlens=d["cu_seqlens"], **kw)
    torch.cuda.synchronize()
    return o, ST, sn


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 128), (128, 64)])
@pytest.mark.parametrize("E,T", [(1, 300), (2, 257), (3, 640)])
def test_snapshots_match_oracle_prefix_states(io, dk, dv, E, T):
    x = inputs.make_prefill(B=2, T=T, H=3, dk=dk, dv=dv, io=io, seed=300 + E * 17 + T + dk + dv, s0_std=0.1)
    print("case: snapshots every %d chunks, B=2 T=%d H=3 dk=%d dv=%d %s" % (E, T, dk, dv, io), flush=True)
    o, ST, sn = _snap(x, E)
    n_snap = (T - 1) // (E * 64)
    assert tuple(sn.shape) == (2, n_snap, 3, dv, dk)
    for s in range(2):
        for j in range(1, n_snap + 1):
            ref = _prefix_state(x, s, j * E * 64)
            err = oracle.max_rel_err(f64(sn[s, j - 1]), ref)
            assert err < TOL[io], (s, j, err)
    # the outputs and the final state are those of the plain call
    d = _dev(x)
    o2, ST2 = gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"])
    torch.cuda.synchronize()
    assert oracle.max_rel_err(f64(o), f64(o2)) < 1e-5
    assert oracle.max_rel_err(f64(ST), f64(ST2)) < 1e-5


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_snapshots_ragged_and_untouched_rows(io):
    lens = [0, 1, 64, 65, 200, 130]
    x = inputs.make_prefill(B=1, T=0, H=2, dk=128, dv=128, io=io, seed=41, s0_std=0.05, lengths=lens)
    print("case: ragged snapshots lens=%s %s" % (lens, io), flush=True)
    T = int(sum(lens))
    n_snap = (T - 1) // 64
    d = _dev(x)
    sn = torch.full((len(lens), n_snap, 2, 128, 128), float("nan"), device="cuda")
    o, ST, sn = gdn.gdn_chunk_prefill_snapshots(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], snap_every=1,
                                                cu_seqlens=d["cu_seqlens"], snaps=sn)
    torch.cuda.synchronize()
    cu = x["cu_seqlens"].tolist()
    for s, n in enumerate(lens):
        taken = (n - 1) // 64 if n > 0 else 0
        for j in range(1, taken + 1):
            seq = {k: x[k][:, cu[s]:cu[s] + j * 64] for k in TOKEN}
            _, ref = oracle.recurrence(*(f64(seq[k]) for k in TOKEN), f64(x["S0"][s:s + 1]))
            assert oracle.max_rel_err(f64(sn[s, j - 1]), ref[0]) < TOL[io], (s, j)
        assert torch.isnan(sn[s, taken:]).all(), s   # past the sequence's last snapshot: untouched
    o_ref, ST_ref = oracle.recurrence(*(f64(x[k]) for k in TOKEN), f64(x["S0"]), cu_seqlens=cu)
    assert oracle.max_rel_err(f64(o), o_ref) < TOL[io]
    assert oracle.max_rel_err(f64(ST), ST_ref) < TOL[io]


def test_snapshots_stay_sequential_where_the_automatic_plan_splits():
    """A split would not form the states inside segments: on a prompt whose plain call the automatic plan
    splits (T=4133, two heads), the snapshot call still takes the sequential form and every snapshot is right."""
    assert gdn.gdn_chunk_prefill_plan(1, 4133, 2, 128, 128, 0, gdn.GDN_BF16)[1] > 1
    x = inputs.make_prefill(B=1, T=4133, H=2, dk=128, dv=128, io="bf16", seed=43, s0_std=0.05)
    print("case: snapshots where the automatic plan splits", flush=True)
    o, ST, sn = _snap(x, 16)
    assert sn.shape[1] == 4
    for j in range(1, sn.shape[1] + 1):
        assert oracle.max_rel_err(f64(sn[0, j - 1]), _prefix_state(x, 0, j * 1024)) < TOL["bf16"], j
    o_ref, ST_ref = oracle.recurrence(*(f64(x[k]) for k in TOKEN), f64(x["S0"]))
    assert oracle.max_rel_err(f64(o), o_ref) < TOL["bf16"]
    assert oracle.max_rel_err(f64(ST), ST_ref) < TOL["bf16"]


def test_snapshots_full_size_one_launch():
    """T=10240, H=16, bf16 (the one-launch form), a snapshot every 2048 tokens."""
    w = inputs.WORKLOADS["prefill_10k_bf16"]
    x = inputs.make_workload("prefill_10k_bf16")
    print("case: %s, snapshots every 32 chunks" % w.name, flush=True)
    o, ST, sn = _snap(x, 32)
    assert sn.shape[1] == 4
    for j in range(1, 5):
        assert oracle.max_rel_err(f64(sn[0, j - 1]), _prefix_state(x, 0, j * 2048)) < TOL["bf16"], j
    o_ref, ST_ref = oracle.recurrence(*(f64(x[k]) for k in TOKEN), f64(x["S0"]))
    assert oracle.max_rel_err(f64(o), o_ref) < TOL["bf16"]
    assert oracle.max_rel_err(f64(ST), ST_ref) < TOL["bf16"]


def test_no_snapshot_inside_a_short_prompt():
    x = inputs.make_prefill(B=1, T=64, H=2, dk=64, dv=64, io="f32", seed=47, s0_std=0.05)
    o, ST, sn = _snap(x, 1)
    assert sn.shape[1] == 0
    o_ref, ST_ref = oracle.recurrence(*(f64(x[k]) for k in TOKEN), f64(x["S0"]))
    assert oracle.max_rel_err(f64(ST), ST_ref) < TOL["f32"]


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("flags", [0, gdn.GDN_QK_L2NORM | gdn.GDN_GATE_LOGITS])
def test_snapshots_ex_grouped_with_input_transforms(io, flags):
    """Grouped key heads (4 value heads over 2) and, in one case, unnormalised q, k and gate logits: every snapshot
    against the oracle's state of that prefix under the same transforms."""
    print("case: snapshots_ex", io, flags, flush=True)
    raw = bool(flags)
    x = inputs.make_prefill(B=2, T=300, H=4, H_k=2, dk=128, dv=128, io=io, seed=820 + flags, s0_std=0.05, raw=raw)
    d = _dev(x)
    o, ST, sn = gdn.gdn_chunk_prefill_snapshots_ex(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], snap_every=2,
                                                   flags=flags)
    torch.cuda.synchronize()
    kw = dict(qk_l2norm=raw, gate_logits=raw)
    o_ref, ST_ref = oracle.recurrence_ex(*(f64(x[k]) for k in TOKEN), f64(x["S0"]), **kw)
    assert oracle.max_rel_err(f64(o), o_ref) < TOL[io]
    assert oracle.max_rel_err(f64(ST), ST_ref) < TOL[io]
    assert sn.shape[1] == (300 - 1) // 128
    for s in range(2):
        for j in range(sn.shape[1]):
            t = (j + 1) * 128
            _, S = oracle.recurrence_ex(*(f64(x[k][s:s + 1, :t]) for k in TOKEN), f64(x["S0"][s:s + 1]), **kw)
            e = oracle.max_rel_err(f64(sn[s, j]), S[0])
            assert e < TOL[io], (s, j, e)


def test_snapshots_ex_full_size_one_launch():
    """T=10240, 16 heads over 8 key heads, bf16, with the input transforms: the one-launch form's snapshot variant."""
    flags = gdn.GDN_QK_L2NORM | gdn.GDN_GATE_LOGITS
    x = inputs.make_prefill(B=1, T=10240, H=16, H_k=8, dk=128, dv=128, io="bf16", seed=821, s0_std=0.02, g_shift=-2.0,
                            raw=True)
    d = _dev(x)
    o, ST, sn = gdn.gdn_chunk_prefill_snapshots_ex(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], snap_every=40,
                                                   flags=flags)
    torch.cuda.synchronize()
    kw = dict(qk_l2norm=True, gate_logits=True)
    o_ref, ST_ref = oracle.recurrence_ex(*(f64(x[k]) for k in TOKEN), f64(x["S0"]), **kw)
    assert oracle.max_rel_err(f64(o), o_ref) < 2e-2 and oracle.max_rel_err(f64(ST), ST_ref) < 2e-2
    _, S = oracle.recurrence_ex(*(f64(x[k][:, :40 * 64 * 2]) for k in TOKEN), f64(x["S0"]), **kw)
    assert oracle.max_rel_err(f64(sn[0, 1]), S[0]) < 2e-2
