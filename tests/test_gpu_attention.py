"""GPU parity of the causal attention prefill (gdn_attention_prefill, through the C ABI)
against the fp64 oracle (``oracle.attention.causal_attention``).

bf16 q, k, v and o with fp32 softmax and accumulation; the bar is the bf16 one of
the other parity tests: max|x - ref| / max|ref| < 2e-2 per output tensor.  At the
full timed size the oracle is evaluated on sampled query rows (every head).
"""
import numpy as np
import pytest
import torch

import paper_2607_14568_amd as gdn
from oracle import attention as att
from paper_2607_14568_amd import inputs

pytestmark = pytest.mark.gpu
TOL = 2e-2
f64 = inputs.as_f64


def _rel(x, ref):
    return float(np.abs(x - ref).max() / np.abs(ref).max())


def _check(B, T, H, Hkv, d, seed, scale=None, rows=None):
    label = "attention B=%d T=%d H=%d H_kv=%d d=%d" % (B, T, H, Hkv, d)
    print("case:", label, flush=True)
    x = inputs.make_attention(B, T, H, Hkv, d, seed)
    sc = 1.0 / d ** 0.5 if scale is None else scale
    o = gdn.gdn_attention_prefill(x["q"].cuda(), x["k"].cuda(), x["v"].cuda(), scale=sc)
    torch.cuda.synchronize()
    ref = att.causal_attention(f64(x["q"]), f64(x["k"]), f64(x["v"]), sc, rows=rows)
    got = f64(o) if rows is None else f64(o)[:, rows]
    e = _rel(got, ref)
    print("  max rel err o=%.3e" % e, flush=True)
    assert np.isfinite(f64(o)).all()
    assert e < TOL, (label, e)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("T", [1, 63, 64, 65, 127, 128, 129, 300])
def test_attention_shapes_and_tails(d, T):
    _check(2, T, 4, 2, d, seed=700 + T + d)


@pytest.mark.parametrize("H,Hkv", [(4, 4), (4, 1), (6, 2)])
def test_attention_grouped_heads(H, Hkv):
    _check(1, 700, H, Hkv, 128, seed=710 + H + Hkv)


def test_attention_sharp_scores():
    """A large scale: softmax close to one-hot, the running max changing often."""
    _check(1, 500, 2, 1, 128, seed=720, scale=1.5)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("scale", [0.0, -0.1])
def test_attention_nonpositive_scale(d, scale):
    """scale = 0 (uniform weights over each prefix) and scale < 0 (the largest
    scaled score is the smallest raw one)."""
    _check(1, 300, 2, 1, d, seed=722 + d, scale=scale)


@pytest.mark.parametrize("growth", [5.0, 20.0])
@pytest.mark.parametrize("B,H", [(1, 2), (4, 64)])
def test_attention_rising_scores(growth, B, H):
    """Scores that rise along the keys by `growth` (log2 units) per 64-key block, on
    top of random ones: the softmax's reference maximum lags the running maximum
    (growth 5) or moves at every block (growth 20).  B = 4, H = 64 is a grid with
    two query tiles per wave."""
    T, d = 400, 128
    if H == 64:
        assert (T + 127) // 128 * B * H >= _wgs_for_two_tiles()
    print("case: attention rising scores growth=%g B=%d H=%d" % (growth, B, H), flush=True)
    x = inputs.make_attention(B, T, H, 1, d, seed=724)
    step = growth / (64 * np.log2(np.e))   # raw score added per key position
    j = torch.arange(T, dtype=torch.float64)
    # q . k_j = j step plus a small random part
    q = 1.0 + 0.1 * x["q"].double()
    k = (j * step / d)[None, :, None, None] + 0.1 * x["k"].double()
    qb, kb = q.to(torch.bfloat16), k.to(torch.bfloat16)
    o = gdn.gdn_attention_prefill(qb.cuda(), kb.cuda(), x["v"].cuda(), scale=1.0)
    torch.cuda.synchronize()
    ref = att.causal_attention(f64(qb), f64(kb), f64(x["v"]), 1.0)
    e = _rel(f64(o), ref)
    print("  max rel err o=%.3e" % e, flush=True)
    assert np.isfinite(f64(o)).all()
    assert e < TOL, e


def test_attention_2k():
    _check(1, 2048, 16, 8, 128, seed=721)


def test_attention_full_size_sampled_rows():
    """The timed shape: T=10240, 16 query heads over 8 key/value heads, d=128; 96 sampled query rows."""
    rows = sorted(set([0, 1, 63, 64, 127, 128, 5000, 10239] + list(np.random.default_rng(5).integers(0, 10240, 88))))
    _check(1, 10240, 16, 8, 128, seed=722, rows=rows)


def test_attention_deterministic_and_grouped_equals_repeated_heads():
    x = inputs.make_attention(1, 333, 4, 2, 128, seed=730)
    q, k, v = x["q"].cuda(), x["k"].cuda(), x["v"].cuda()
    a = gdn.gdn_attention_prefill(q, k, v)
    b = gdn.gdn_attention_prefill(q, k, v)
    c = gdn.gdn_attention_prefill(q, k.repeat_interleave(2, dim=2).contiguous(), v.repeat_interleave(2, dim=2).contiguous())
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(a, c)


def _wgs_for_two_tiles():
    """Workgroups from which the d = 128 kernel takes two query tiles per wave."""
    return 4 * torch.cuda.get_device_properties(0).multi_processor_count


@pytest.mark.parametrize("T", [1, 17, 65, 300])
def test_attention_two_query_tiles_per_wave(T):
    """A grid of at least four workgroups per CU at d = 128 (the form with two 16-query tiles per
    wave), with one-block and ragged tails."""
    nqb = (T + 127) // 128
    B, H = 8, 64
    while nqb * B * H < _wgs_for_two_tiles():
        B *= 2
    _check(B, T, H, 16, 128, seed=730 + T)


@pytest.mark.parametrize("d,H,Hkv", [(64, 4, 2), (128, 4, 2), (128, 64, 16)])
def test_attention_packed_sequences(d, H, Hkv):
    """Sequences packed with cu_seqlens (empty, one-token, block-edge and ragged lengths) attend only within
    themselves: each compared with the oracle over that sequence alone.  At 64 heads the grid takes the
    form with two query tiles per wave."""
    lens = [0, 1, 128, 129, 300, 64, 0, 777, 5]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cu[-1])
    if H == 64:
        assert ((T + 127) // 128 + len(lens)) * H >= _wgs_for_two_tiles()
    print("case: attention packed lengths %s d=%d H=%d" % (lens, d, H), flush=True)
    x = inputs.make_attention(1, T, H, Hkv, d, seed=740 + d + H)
    sc = 1.0 / d ** 0.5
    o = gdn.gdn_attention_prefill(x["q"].cuda(), x["k"].cuda(), x["v"].cuda(), scale=sc,
                                  cu_seqlens=torch.from_numpy(cu).cuda())
    torch.cuda.synchronize()
    got = f64(o)
    q, k, v = f64(x["q"]), f64(x["k"]), f64(x["v"])
    worst = 0.0
    for s0, s1 in zip(cu[:-1], cu[1:]):
        if s1 > s0:
            ref = att.causal_attention(q[:, s0:s1], k[:, s0:s1], v[:, s0:s1], sc)
            worst = max(worst, _rel(got[:, s0:s1], ref))
    print("  max rel err o=%.3e" % worst, flush=True)
    assert worst < TOL
