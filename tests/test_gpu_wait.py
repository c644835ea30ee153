"""The one-launch prefill's bounded wait reports failure instead of computing on unpublished terms.

GDN_TEST_WITHHOLD makes the chunk-terms workgroups of the one-launch form publish nothing and the chain
give up after 1024 polls, from the host: every kernel exits normally, the outputs are NaN and
gdn_workspace_status reports GDN_ERR_WAIT once (then the word is clear).  The same workspace then serves a
normal call, checked against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_14568_amd as gdn
from paper_2607_14568_amd import inputs

pytestmark = pytest.mark.gpu

f = inputs.as_f64


def _inputs(seed):
    # bf16, 2 heads, 300 tokens: the sequential form, in one launch (16 chain workgroups leave CUs free)
    x = inputs.make_prefill(B=1, T=300, H=2, dk=128, dv=128, io="bf16", seed=seed, s0_std=0.02)
    return x, {k: (v.cuda() if v is not None else None) for k, v in x.items()}


def _call(d, ws, flags):
    return gdn.gdn_chunk_prefill_ex(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"],
                                    flags=gdn.GDN_PLAN_SEQUENTIAL | flags, workspace=ws)


def test_withheld_terms_are_reported_and_the_workspace_recovers():
    x, d = _inputs(31)
    need = gdn.gdn_chunk_prefill_workspace_bytes_ex(1, 300, 2, 128, 128, 64, 0, gdn.GDN_BF16, gdn.GDN_PLAN_SEQUENTIAL)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    gdn.gdn_workspace_status(ws)   # whatever the fresh workspace held: not this process's tag
    o, S_T = _call(d, ws, gdn.GDN_TEST_WITHHOLD)
    torch.cuda.synchronize()
    assert torch.isnan(o.float()).all(), "outputs after a failed wait must be NaN"
    assert torch.isnan(S_T).all(), "the final state after a failed wait must be NaN"
    with pytest.raises(gdn.GdnError) as e:
        gdn.gdn_workspace_status(ws)
    assert e.value.status == gdn.GDN_ERR_WAIT
    gdn.gdn_workspace_status(ws)   # reported once, then clear
    # the same workspace, a normal call: published terms, correct results, nothing reported
    o, S_T = _call(d, ws, 0)
    torch.cuda.synchronize()
    gdn.gdn_workspace_status(ws)
    ro, rs = oracle.recurrence(f(x["q"]), f(x["k"]), f(x["v"]), f(x["g"]), f(x["beta"]), f(x["S0"]))
    assert oracle.max_rel_err(f(o), ro) < 2e-2
    assert oracle.max_rel_err(f(S_T), rs) < 2e-2


def test_normal_calls_report_nothing():
    x, d = _inputs(32)
    need = gdn.gdn_chunk_prefill_workspace_bytes_ex(1, 300, 2, 128, 128, 64, 0, gdn.GDN_BF16, gdn.GDN_PLAN_SEQUENTIAL)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for _ in range(3):
        o, S_T = _call(d, ws, 0)
    gdn.gdn_workspace_status(ws)
    assert np.isfinite(f(o)).all() and np.isfinite(f(S_T)).all()
