"""GPU parity of the segment-parallel prefill (through the C ABI) against the fp64 oracle.

The chunk map of section 3.2 is affine in the state, so a sequence cut into
segments at chunk boundaries gives the same o and S_T as the sequential chain
(up to rounding).  These cases force the narrow split per call
(gdn_chunk_prefill_ex with GDN_PLAN_SEGMENTED and a segment count) and compare with the oracle at the bars of the other prefill tests
(max|x - ref| / max|ref|: 2e-4 fp32 io, 2e-2 bf16 io).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_14568_amd as gdn
from paper_2607_14568_amd import inputs

pytestmark = pytest.mark.gpu
TOL = {"f32": 2e-4, "bf16": 2e-2}
IO = {"f32": gdn.GDN_F32, "bf16": gdn.GDN_BF16}
f64 = inputs.as_f64


SEG = gdn.GDN_PLAN_SEGMENTED


def _dev(x):
    return {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in x.items()}


def _ref(x, scale=1.0):
    return oracle.recurrence(f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["g"]), f64(x["beta"]),
                             f64(x["S0"]), scale=scale)


def _prefill(d, P, **kw):
    """The prefill with the narrow segment-parallel plan forced to P segments (P = 1: the sequential form)."""
    flags, segs = (gdn.GDN_PLAN_SEQUENTIAL, 0) if P == 1 else (SEG, P)
    return gdn.gdn_chunk_prefill_ex(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], flags=flags, segments=segs, **kw)


def _check(x, io, label, P, scale=1.0, **kw):
    print("case:", label, flush=True)
    d = _dev(x)
    o, ST = _prefill(d, P, scale=scale, **kw)
    torch.cuda.synchronize()
    o_ref, ST_ref = _ref(x, scale)
    eo, es = oracle.max_rel_err(f64(o), o_ref), oracle.max_rel_err(f64(ST), ST_ref)
    print("  max rel err o=%.3e S_T=%.3e" % (eo, es), flush=True)
    assert np.isfinite(f64(o)).all() and np.isfinite(f64(ST)).all()
    assert eo < TOL[io], (label, eo)
    assert es < TOL[io], (label, es)
    return o, ST


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
@pytest.mark.parametrize("P,T", [(2, 130), (3, 700), (5, 1000), (8, 64 * 16 + 17)])
def test_segmented_matches_oracle(io, dk, dv, P, T):
    """Several segment counts, every (dk, dv), ragged tails inside the last chunk and segment, B=2, carried S0."""
    x = inputs.make_prefill(B=2, T=T, H=3, dk=dk, dv=dv, io=io, seed=1000 + P * 31 + T + dk + dv, s0_std=0.1)
    _check(x, io, "segments=%d B=2 T=%d H=3 dk=%d dv=%d %s" % (P, T, dk, dv, io), P)


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_segmented_no_initial_state_and_scale(io):
    x = inputs.make_prefill(B=1, T=777, H=2, dk=128, dv=128, io=io, seed=7)
    assert x["S0"] is None
    _check(x, io, "segments=4 S0=None scale", 4, scale=128 ** -0.5)


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("case", ["alpha0", "alpha1", "beta0", "beta1"])
def test_segmented_extreme_gates(io, case):
    """alpha = 0 (each segment's transition vanishes), alpha = 1, beta = 0 (pure decay: the
    transition is a scalar), beta = 1."""
    x = inputs.make_prefill(B=1, T=500, H=2, dk=128, dv=64, io=io, seed=13, s0_std=0.1)
    if case == "alpha0":
        x["g"].fill_(-1e4)
    elif case == "alpha1":
        x["g"].zero_()
    elif case == "beta0":
        x["beta"].zero_()               # pure decay of S0; milder decay keeps
        x["g"].mul_(0.05)               # exp(sum g) S0 inside the fp32 range
    else:
        x["beta"].fill_(1.0)
    _check(x, io, "segments=3 " + case, 3)


def test_segmented_many_short_segments():
    """64 requested on 70 chunks: segments of 2 chunks (35 of them), the longest scan."""
    x = inputs.make_prefill(B=1, T=64 * 70 + 5, H=2, dk=64, dv=64, io="f32", seed=17, s0_std=0.1)
    _check(x, "f32", "segments=64 T=4485", 64)


def test_segmented_in_place_state():
    x = inputs.make_prefill(B=2, T=400, H=2, dk=64, dv=128, io="f32", seed=19, s0_std=0.05)
    o_ref, ST_ref = _ref(x)
    d = _dev(x)
    S = d["S0"].clone()
    d["S0"] = S
    o, ST = _prefill(d, 3, S_T=S)
    torch.cuda.synchronize()
    assert ST.data_ptr() == S.data_ptr()
    assert oracle.max_rel_err(f64(S), ST_ref) < TOL["f32"]
    assert oracle.max_rel_err(f64(o), o_ref) < TOL["f32"]


def test_headline_shape_plans():
    """16 heads at T=10240 stay sequential in both io types (the split forms' extra work outweighs the CUs
    they would fill); 8 bf16 heads take the wide form, 2 take the narrow split."""
    assert gdn.gdn_chunk_prefill_plan(1, 10240, 16, 128, 128, 0, gdn.GDN_BF16) == (gdn.GDN_PLAN_SEQUENTIAL, 1)
    assert gdn.gdn_chunk_prefill_plan(1, 10240, 16, 128, 128, 0, gdn.GDN_F32) == (gdn.GDN_PLAN_SEQUENTIAL, 1)
    assert gdn.gdn_chunk_prefill_plan(1, 10240, 8, 128, 128, 0, gdn.GDN_BF16) == (gdn.GDN_PLAN_WIDE, 16)
    assert gdn.gdn_chunk_prefill_plan(1, 10240, 2, 128, 128, 0, gdn.GDN_BF16)[0] == gdn.GDN_PLAN_SEGMENTED


def test_segmented_agrees_with_sequential():
    """The same inputs through both forms: equal to bf16 rounding of o, and close in S_T."""
    x = inputs.make_prefill(B=1, T=2000, H=2, dk=128, dv=128, io="bf16", seed=23, s0_std=0.05)
    d = _dev(x)
    res = {}
    for P in (1, 4):
        o, ST = _prefill(d, P)
        torch.cuda.synchronize()
        res[P] = (o, ST)
    assert oracle.max_rel_err(f64(res[4][0]), f64(res[1][0])) < 1e-2
    assert oracle.max_rel_err(f64(res[4][1]), f64(res[1][1])) < 1e-2


def test_segmented_bitwise_deterministic_and_every_output_written():
    x = inputs.make_prefill(B=1, T=1333, H=2, dk=128, dv=128, io="bf16", seed=29, s0_std=0.05)
    d = _dev(x)
    outs = []
    for _ in range(2):
        o = torch.full_like(d["v"], float("nan"))
        ST = torch.full_like(d["S0"], float("nan"))
        _prefill(d, 5, o=o, S_T=ST)
        torch.cuda.synchronize()
        assert torch.isfinite(o).all() and torch.isfinite(ST).all()
        outs.append((o.clone(), ST.clone()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


def test_segmented_workspace_too_small_splits_less():
    """A workspace sized for the sequential form: the call must still be right (it splits less)."""
    x = inputs.make_prefill(B=1, T=900, H=2, dk=128, dv=128, io="bf16", seed=31, s0_std=0.05)
    need = gdn.gdn_chunk_prefill_workspace_bytes_ex(1, 900, 2, 128, 128, 64, 0, gdn.GDN_BF16, gdn.GDN_PLAN_SEQUENTIAL, 0)
    assert gdn.gdn_chunk_prefill_workspace_bytes_ex(1, 900, 2, 128, 128, 64, 0, gdn.GDN_BF16, SEG, 4) > need
    assert gdn.gdn_chunk_prefill_plan(1, 900, 2, 128, 128, 0, gdn.GDN_BF16, SEG, 4, need) == (gdn.GDN_PLAN_SEQUENTIAL, 1)
    ws = torch.full((need,), 0xFF, dtype=torch.uint8, device="cuda")
    _check(x, "bf16", "segments=4, sequential-size workspace", 4, workspace=ws)


@pytest.mark.parametrize("io,H", [("bf16", 2), ("bf16", 4), ("f32", 2)])
def test_automatic_split_long_prompt(io, H):
    """T=10240, d=128 with few heads: the automatic plan splits (on a 256-CU device; the
    workspace function assumes one).  Full-size parity against the oracle."""
    x = inputs.make_prefill(B=1, T=10240, H=H, dk=128, dv=128, io=io, seed=37 + H,
                            s0_std=0.02, g_shift=2.0)
    assert gdn.gdn_chunk_prefill_workspace_bytes(1, 10240, H, 128, 128, 64, 0, IO[io]) > \
        gdn.gdn_chunk_prefill_workspace_bytes_ex(1, 10240, H, 128, 128, 64, 0, IO[io], gdn.GDN_PLAN_SEQUENTIAL, 0)
    form, P = gdn.gdn_chunk_prefill_plan(1, 10240, H, 128, 128, 0, IO[io])
    assert form == SEG and P > 1, (form, P)
    print("case: automatic split T=10240 H=%d %s" % (H, io), flush=True)
    d = _dev(x)
    o, ST = gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"])
    torch.cuda.synchronize()
    o_ref, ST_ref = _ref(x)
    assert oracle.max_rel_err(f64(o), o_ref) < TOL[io] and oracle.max_rel_err(f64(ST), ST_ref) < TOL[io]
