"""Full-length parity with the state carried across many chunks (alpha near 1).

The timed 10k workload's gates (g = -softplus(N(0,1)+2)) decay the state by about e^-140 per 64-token chunk, so
there nothing survives a chunk.  Here g = -softplus(N(0,1) - 6) (alpha ~ 0.9975 per token, ~0.85 per chunk) and
g = 0 with small beta (no decay at all) carry the state over the whole prompt, through the one-launch sequential
chain at 16 heads (bf16 operands of S_c over 160 chunks) and the automatic segmented form at 2 heads (the
entering states composed across segments), in bf16 and fp32.  Parity per tensor and per (sequence, head).
"""
import pytest
import torch

import oracle
import paper_2607_14568_amd as gdn
import parity
from paper_2607_14568_amd import inputs

pytestmark = pytest.mark.gpu
f64 = inputs.as_f64
PLANS = {"seq": gdn.GDN_PLAN_SEQUENTIAL, "auto": 0}


def _case(io, H, gates, seed):
    x = inputs.make_prefill(B=1, T=10240, H=H, dk=128, dv=128, io=io, seed=seed, s0_std=0.02, g_shift=-6.0)
    if gates == "alpha1":   # no decay, small writes
        x["g"][:] = 0.0
        x["beta"] *= 0.05
    return x


@pytest.mark.parametrize("gates", ["slow", "alpha1"])
@pytest.mark.parametrize("io,H,plan", [("bf16", 16, "seq"), ("f32", 16, "seq"), ("bf16", 2, "auto"),
                                       ("f32", 2, "auto")])
def test_long_memory_full_length(io, H, plan, gates):
    x = _case(io, H, gates, 700 + H + (1 if io == "f32" else 0) + (2 if gates == "alpha1" else 0))
    form, P = gdn.gdn_chunk_prefill_plan(1, 10240, H, 128, 128, 0, gdn.GDN_BF16 if io == "bf16" else gdn.GDN_F32,
                                         PLANS[plan])
    if plan == "auto":
        assert P > 1, "two heads at T=10240 take a segmented form"
    label = "long memory %s T=10240 H=%d %s (form %d, %d segments)" % (gates, H, io, form, P)
    print("case:", label, flush=True)
    d = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in x.items()}
    o, ST = gdn.gdn_chunk_prefill_ex(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], flags=PLANS[plan])
    torch.cuda.synchronize()
    ro, rs = oracle.recurrence(f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["g"]), f64(x["beta"]), f64(x["S0"]))
    parity.check(f64(o), ro, f64(ST), rs, parity.TOL[io], label)
