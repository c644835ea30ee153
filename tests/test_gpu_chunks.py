"""GPU parity of the prefill at chunk lengths 16, 32 and 128 (the generic path) against the fp64 oracle.

Section 3.2 leaves the chunk length free: the chunked form equals the token-by-token recurrence at every
chunk length, so each length must match the oracle to the io type's bar, per output tensor and per
(sequence, head) slice, with sequences of 1, C - 1, C and C + 1 tokens, ragged packing, grouped key heads with
the input transforms, the limiting gates, and the 10k-token 16-head prompt at chunk 128.  Different chunk
lengths (64 included) must agree with each other.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_14568_amd as gdn
import parity
from paper_2607_14568_amd import inputs

pytestmark = pytest.mark.gpu
f64 = inputs.as_f64
CHUNKS = (16, 32, 128)


def _dev(x):
    return {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in x.items()}


def _ref(x, scale=1.0, cu=None):
    return oracle.recurrence(f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["g"]), f64(x["beta"]), f64(x["S0"]),
                             cu_seqlens=cu, scale=scale)


def _run(x, C, **kw):
    d = _dev(x)
    o, ST = gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], chunk=C,
                                  cu_seqlens=d.get("cu_seqlens"), **kw)
    torch.cuda.synchronize()
    return o, ST


@pytest.mark.parametrize("io", ["bf16", "f32"])
@pytest.mark.parametrize("C", CHUNKS)
def test_chunk_lengths_match_oracle(C, io):
    for d in (64, 128):
        for T in (1, C - 1, C, C + 1, 2 * C + 5):
            label = "chunk=%d %s d=%d T=%d" % (C, io, d, T)
            print("case:", label, flush=True)
            x = inputs.make_prefill(B=2, T=T, H=3, dk=d, dv=d, io=io, seed=100 * C + T + d, s0_std=0.05)
            o, ST = _run(x, C)
            ro, rs = _ref(x)
            parity.check(f64(o), ro, f64(ST), rs, parity.TOL[io], label)


@pytest.mark.parametrize("io", ["bf16", "f32"])
@pytest.mark.parametrize("C", CHUNKS)
def test_chunk_lengths_ragged(C, io):
    lengths = [0, 1, C - 1, C, C + 1, 3 * C + 2, 5]
    x = inputs.make_prefill(B=1, T=0, H=2, dk=128, dv=64, io=io, seed=7 + C, s0_std=0.05, lengths=lengths)
    cu = x["cu_seqlens"].numpy()
    label = "ragged chunk=%d %s lengths=%s" % (C, io, lengths)
    print("case:", label, flush=True)
    o, ST = _run(x, C)
    ro, rs = _ref(x, cu=cu)
    parity.check(f64(o), ro, f64(ST), rs, parity.TOL[io], label, cu_seqlens=cu)
    # the empty sequence keeps its initial state
    assert np.array_equal(f64(ST)[0], f64(x["S0"])[0])


@pytest.mark.parametrize("C", (32, 128))
def test_chunk_lengths_grouped_with_transforms(C):
    x = inputs.make_prefill(B=1, T=3 * C + 9, H=4, H_k=2, dk=128, dv=128, io="bf16", seed=11 + C, s0_std=0.02,
                            raw=True)
    d = _dev(x)
    flags = gdn.GDN_QK_L2NORM | gdn.GDN_GATE_LOGITS
    print("case: grouped 4 over 2 heads with the input transforms, chunk=%d" % C, flush=True)
    o, ST = gdn.gdn_chunk_prefill_ex(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], flags=flags, chunk=C,
                                     scale=0.5)
    torch.cuda.synchronize()
    ro, rs = oracle.recurrence_ex(f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["g"]), f64(x["beta"]),
                                  f64(x["S0"]), qk_l2norm=True, gate_logits=True, scale=0.5)
    parity.check(f64(o), ro, f64(ST), rs, parity.TOL["bf16"], "grouped ex chunk=%d" % C)


@pytest.mark.parametrize("case", ["alpha0", "alpha1", "beta0"])
def test_chunk_lengths_limiting_gates(case):
    x = inputs.make_prefill(B=1, T=150, H=2, dk=64, dv=64, io="f32", seed=3, s0_std=0.1)
    if case == "alpha0":
        x["g"][:] = -1e4
    elif case == "alpha1":
        x["g"][:] = 0.0
    else:   # pure decay of S0: a mild decay, so the state stays well inside fp32's range
        x["beta"][:] = 0.0
        x["g"][:] = -0.01
    ro, rs = _ref(x)
    for C in CHUNKS:
        label = "%s chunk=%d" % (case, C)
        print("case:", label, flush=True)
        o, ST = _run(x, C)
        parity.check(f64(o), ro, f64(ST), rs, parity.TOL["f32"], label)


def test_chunk_lengths_agree_with_each_other():
    """The result does not depend on the chunk length: 16, 32, 64 and 128 agree to rounding."""
    x = inputs.make_prefill(B=1, T=700, H=2, dk=128, dv=128, io="f32", seed=21, s0_std=0.05, g_shift=-2.0)
    res = {C: _run(x, C) for C in (16, 32, 64, 128)}
    for C in (16, 32, 128):
        assert oracle.max_rel_err(f64(res[C][0]), f64(res[64][0])) < 2e-4, C
        assert oracle.max_rel_err(f64(res[C][1]), f64(res[64][1])) < 2e-4, C


def test_chunk_128_in_place_and_deterministic():
    x = inputs.make_prefill(B=1, T=300, H=2, dk=128, dv=128, io="bf16", seed=5, s0_std=0.1)
    ro, rs = _ref(x)
    d = _dev(x)
    S = d["S0"].clone()
    o1, _ = gdn.gdn_chunk_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], S, S_T=S, chunk=128)
    torch.cuda.synchronize()
    parity.check(f64(o1), ro, f64(S), rs, parity.TOL["bf16"], "chunk=128 in place")
    o2, S2 = _run(x, 128)
    o3, S3 = _run(x, 128)
    assert torch.equal(o2, o3) and torch.equal(S2, S3)


def test_chunk_128_full_size():
    """T=10240, H=16, d=128, bf16 at chunk 128, and the slow-decay variant (state carried across chunks)."""
    for name in ("prefill_10k_bf16", "prefill_10k_bf16_slow"):
        x = inputs.make_workload(name)
        print("case: %s at chunk=128" % name, flush=True)
        o, ST = _run(x, 128)
        ro, rs = _ref(x)
        parity.check(f64(o), ro, f64(ST), rs, parity.TOL["bf16"], name + " chunk=128")
