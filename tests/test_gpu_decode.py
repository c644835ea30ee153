"""GPU parity of the decode step (through the C ABI) against the fp64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_14568_amd as gdn
from paper_2607_14568_amd import inputs

pytestmark = pytest.mark.gpu
f64 = inputs.as_f64


def _replay(y, steps, io_tol):
    """Run `steps` decode steps (token i % pool) and compare every step's o and the final S."""
    pool = y["q"].shape[0]
    d = {k: v.cuda() for k, v in y.items()}
    S = d["S"].clone()
    S_ref = f64(y["S"])
    worst = 0.0
    for i in range(steps):
        j = i % pool
        o = gdn.gdn_decode_step(d["q"][j], d["k"][j], d["v"][j], d["g"][j], d["beta"][j], S)
        o_ref, S_ref = oracle.decode_step(f64(y["q"][j]), f64(y["k"][j]), f64(y["v"][j]), f64(y["g"][j]),
                                          f64(y["beta"][j]), S_ref)
        e = oracle.max_rel_err(f64(o), o_ref)
        worst = max(worst, e)
        assert e < io_tol, (i, e)
    es = oracle.max_rel_err(f64(S), S_ref)
    print("  decode %d steps: worst o err %.3e, final S err %.3e" % (steps, worst, es), flush=True)
    assert es < io_tol
    assert np.isfinite(f64(S)).all()


def test_decode_b64_workload():
    """64 sequences x 16 heads x 128x128 state, fp32; 100 steps of the 1000-step loop."""
    w = inputs.WORKLOADS["decode_b64_f32"]
    print("case: decode_b64_f32", flush=True)
    _replay(inputs.make_workload("decode_b64_f32"), 100, 2e-4)


@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("dk,dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
def test_decode_shapes(io, dk, dv):
    print("case: decode", io, dk, dv, flush=True)
    y = inputs.make_decode(B=5, H=3, dk=dk, dv=dv, io=io, seed=dk + dv, pool=4)
    _replay(y, 12, 2e-4 if io == "f32" else 2e-2)


def test_decode_extreme_gates():
    y = inputs.make_decode(B=4, H=2, dk=128, dv=128, io="f32", seed=9, pool=3)
    y["g"][0].fill_(-1e4)
    y["g"][1].zero_()
    y["beta"][2].zero_()
    _replay(y, 6, 2e-4)


def test_decode_b512_workload():
    """512 sequences x 16 heads (537 MB of state, past the Infinity Cache): 3 steps, every output compared."""
    print("case: decode_b512_f32", flush=True)
    _replay(inputs.make_workload("decode_b512_f32"), 3, 2e-4)
