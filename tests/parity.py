"""Parity assertions shared by the GPU tests.

The bar (max|x - ref| / max|ref|, 2e-4 for fp32 io and 2e-2 for bf16 io) is asserted on each output
tensor as a whole and on every (sequence, head) slice against that slice's own largest reference
value, so that an error confined to one head or one sequence is not hidden by a larger scale
elsewhere.  The 99th percentile of |x - ref| / (|ref| + 1e-3 rms(ref)) is printed for information.
"""
import numpy as np

import oracle

TOL = {"f32": 2e-4, "bf16": 2e-2}


def seq_head_slices(o_shape, cu_seqlens=None):
    """Index tuples of the (sequence, head) slices of o [B, T, H, dv] and of S_T [n, H, dv, dk]."""
    B, T, H = o_shape[:3]
    if cu_seqlens is None:
        o_idx = [(b, slice(None), h) for b in range(B) for h in range(H)]
        s_idx = [(b, h) for b in range(B) for h in range(H)]
    else:
        cu = np.asarray(cu_seqlens)
        o_idx = [(0, slice(int(cu[s]), int(cu[s + 1])), h) for s in range(len(cu) - 1) for h in range(H)]
        s_idx = [(s, h) for s in range(len(cu) - 1) for h in range(H)]
    return o_idx, s_idx


def check(o, o_ref, ST, ST_ref, tol, label, cu_seqlens=None, per_slice=True):
    """Assert the parity bar on o and S_T (numpy fp64 arrays), whole and per (sequence, head)."""
    assert np.isfinite(o).all() and np.isfinite(ST).all(), label
    eo, es = oracle.max_rel_err(o, o_ref), oracle.max_rel_err(ST, ST_ref)
    po, ps = oracle.p99_rel_err(o, o_ref), oracle.p99_rel_err(ST, ST_ref)
    msg = "  max rel err o=%.3e S_T=%.3e  p99 elementwise o=%.3e S_T=%.3e" % (eo, es, po, ps)
    ho = hs = None
    if per_slice:
        o_idx, s_idx = seq_head_slices(o.shape, cu_seqlens)
        ho = oracle.max_rel_err_slices(o, o_ref, o_idx)
        hs = oracle.max_rel_err_slices(ST, ST_ref, s_idx)
        msg += "  per (seq, head) o=%.3e S_T=%.3e" % (ho, hs)
    print(msg, flush=True)
    assert eo < tol and es < tol, (label, eo, es)
    if per_slice:
        assert ho < tol and hs < tol, (label, "per (seq, head)", ho, hs)
    return eo, es
