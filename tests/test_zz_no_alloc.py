"""The allocation-free prefill (gdn_chunk_prefill_noalloc, through the C ABI) against gdn_chunk_prefill_ex.

Both run on the same seeded inputs; gdn_chunk_prefill_ex gets a workspace of the
size the allocation-free call holds, so both take the same plan.  The calls come
in a row, each later one smaller than the one before it, so a later call runs on
scratch that still holds the earlier call's contents.  Bars as the prefill parity
tests (max|x - ref| / max|ref|: 2e-4 fp32 io, 2e-2 bf16 io), against the
workspace call and against the fp64 oracle.
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


def _dev(x):
    return {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in x.items()}


def _pair(x, flags):
    d = _dev(x)
    o1 = torch.full_like(d["v"], float("nan"))
    n = d["S0"].shape[0] if d["S0"] is not None else (d["cu_seqlens"].numel() - 1 if d["cu_seqlens"] is not None
                                                        else d["v"].shape[0])
    H, dv, dk = d["v"].shape[2], d["v"].shape[3], d["q"].shape[3]
    S1 = torch.full((n, H, dv, dk), float("nan"), device="cuda")
    gdn.gdn_chunk_prefill_noalloc(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], flags=flags,
                                  cu_seqlens=d["cu_seqlens"], o=o1, S_T=S1)
    ws = torch.empty(gdn.GDN_NOALLOC_SCRATCH_BYTES, dtype=torch.uint8, device="cuda")
    o2, S2 = gdn.gdn_chunk_prefill_ex(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], flags=flags,
                                      cu_seqlens=d["cu_seqlens"], workspace=ws)
    torch.cuda.synchronize()
    return o1, S1, o2, S2


CASES = [
    # (label, io, flags, input recipe); each smaller than the one before
    ("bf16 B=1 T=4133 H=16 d=128 automatic plan", "bf16", 0,
     dict(B=1, T=4133, H=16, dk=128, dv=128, io="bf16", seed=71, s0_std=0.05)),
    ("bf16 B=1 T=2500 H=8 d=128 sequential plan", "bf16", gdn.GDN_PLAN_SEQUENTIAL,
     dict(B=1, T=2500, H=8, dk=128, dv=128, io="bf16", seed=72, s0_std=0.05)),
    ("f32 ragged lengths 300,0,517,64 H=2 dk=64 dv=128", "f32", 0,
     dict(B=1, T=881, H=2, dk=64, dv=128, io="f32", seed=73, s0_std=0.05, lengths=[300, 0, 517, 64])),
    ("bf16 B=2 T=65 H=2 d=64", "bf16", 0,
     dict(B=2, T=65, H=2, dk=64, dv=64, io="bf16", seed=74, s0_std=0.05)),
]


def test_noalloc_matches_workspace_call_in_a_row():
    for label, io, flags, recipe in CASES:
        print("case:", label, flush=True)
        x = inputs.make_prefill(**recipe)
        o1, S1, o2, S2 = _pair(x, flags)
        eo, es = oracle.max_rel_err(f64(o1), f64(o2)), oracle.max_rel_err(f64(S1), f64(S2))
        print("  vs workspace call: o=%.3e S_T=%.3e bitwise equal: %s" % (
            eo, es, bool(torch.equal(o1, o2) and torch.equal(S1, S2))), flush=True)
        assert torch.isfinite(o1).all() and torch.isfinite(S1).all()
        assert eo < TOL[io] and es < TOL[io], (label, eo, es)
        cu = None if x["cu_seqlens"] is None else x["cu_seqlens"].numpy()
        o_ref, S_ref = oracle.recurrence(f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["g"]), f64(x["beta"]),
                                         f64(x["S0"]), cu_seqlens=cu)
        parity.check(f64(o1), o_ref, f64(S1), S_ref, TOL[io], label + " vs oracle", cu_seqlens=cu)


def test_noalloc_rejects_sizes_beyond_its_scratch():
    """T=32768, H=16, d=128 bf16 needs 104 MiB of workspace in the sequential form: refused, nothing launched."""
    need = gdn.gdn_chunk_prefill_workspace_bytes_ex(1, 32768, 16, 128, 128, 64, 0, gdn.GDN_BF16,
                                                    gdn.GDN_PLAN_SEQUENTIAL, 0)
    assert need > gdn.GDN_NOALLOC_SCRATCH_BYTES
    t = torch.zeros(16, device="cuda")
    p = t.data_ptr()
    st = gdn.lib().gdn_chunk_prefill_noalloc(p, p, p, p, p, None, p, None, 1, 32768, 16, 16, 128, 128, 64, None, 0,
                                             gdn.GDN_BF16, 1.0, 0, 0, None)
    assert st == 3 and b"scratch" in gdn.lib().gdn_last_error_message()
