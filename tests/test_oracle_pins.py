"""Pins of the fp64 oracle against what the paper and the mathematics fix.

The oracle (``oracle.recurrence``) is the plain token-by-token definition of
the gated delta rule (paper, section 2.2 / section 3.2).  Each test below
checks it against something other than itself: a hand-worked example, exact
rational brute force of the matrix form, closed forms of limiting cases,
invariants of the recurrence, and the independent chunked form of section
3.2 at every chunk size.
"""
import math
import os
from fractions import Fraction as Fr

import numpy as np
import pytest

import oracle
from oracle import chunked as ch

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(seed, B=1, T=13, H=2, dk=5, dv=3, s0=True, g_scale=1.0):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, T, H, dk))
    k = rng.standard_normal((B, T, H, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    v = rng.standard_normal((B, T, H, dv))
    beta = 1 / (1 + np.exp(-rng.standard_normal((B, T, H))))
    g = -np.logaddexp(0, g_scale * rng.standard_normal((B, T, H)))
    S0 = rng.standard_normal((B, H, dv, dk)) * 0.5 if s0 else None
    return q, k, v, g, beta, S0


# --------------------------------------------------------------------------- golden
def _read_golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, rhs = line.split(":", 1)
            items = [Fr(x.strip()) for x in rhs.split(",")]
            vals[key.strip()] = items if len(items) > 1 else items[0]
    return vals


def _frac_matrix_recurrence(S0, ks, vs, qs, betas, alphas):
    """Exact rationals, matrix form: S <- alpha S (I - beta k k^T) + beta v k^T."""
    dv, dk = len(S0), len(S0[0])
    S = [row[:] for row in S0]
    outs = []
    for k, v, q, b, a in zip(ks, vs, qs, betas, alphas):
        M = [[(Fr(1) if i == j else Fr(0)) - b * k[i] * k[j] for j in range(dk)] for i in range(dk)]
        S = [[a * sum(S[r][i] * M[i][c] for i in range(dk)) + b * v[r] * k[c] for c in range(dk)]
             for r in range(dv)]
        outs.append([sum(S[r][c] * q[c] for c in range(dk)) for r in range(dv)])
    return outs, S


def test_golden_handworked_example():
    gd = _read_golden("gdn_handworked_dk2_dv2_T3.txt")
    dk, dv, T = int(gd["dk"]), int(gd["dv"]), int(gd["T"])
    rs = lambda x, *shape: np.array([float(y) for y in x]).reshape(shape)
    q = rs(gd["q"], 1, T, 1, dk)
    k = rs(gd["k"], 1, T, 1, dk)
    v = rs(gd["v"], 1, T, 1, dv)
    beta = rs(gd["beta"], 1, T, 1)
    g = np.log(rs(gd["alpha"], 1, T, 1))
    S0 = rs(gd["S0"], 1, 1, dv, dk)
    o, ST = oracle.recurrence(q, k, v, g, beta, S0)
    np.testing.assert_allclose(o.reshape(-1), [float(x) for x in gd["o"]], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(ST.reshape(-1), [float(x) for x in gd["S_T"]], rtol=1e-14, atol=1e-15)
    # the hand derivation itself agrees with exact rational arithmetic
    S0f = [gd["S0"][r * dk:(r + 1) * dk] for r in range(dv)]
    sl = lambda x, n: [x[i * n:(i + 1) * n] for i in range(T)]
    outs, Sf = _frac_matrix_recurrence(S0f, sl(gd["k"], dk), sl(gd["v"], dv), sl(gd["q"], dk),
                                       gd["beta"], gd["alpha"])
    assert [x for row in outs for x in row] == gd["o"]
    assert [x for row in Sf for x in row] == gd["S_T"]


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_brute_force_exact_rationals(seed):
    """Unnormalised rational keys, rational alpha/beta: matrix form in Fractions."""
    rng = np.random.default_rng(seed)
    dk, dv, T = 3, 2, 5
    rq = lambda *s: rng.integers(-16, 17, size=s) / 8.0          # exact in fp64
    k, v, q = rq(T, dk), rq(T, dv), rq(T, dk)
    S0 = rq(dv, dk)
    beta = rng.integers(1, 8, size=T) / 8.0
    g = -rng.uniform(0.05, 2.0, size=T)
    alpha_fp = np.exp(g)                                         # what the oracle uses
    o, ST = oracle.recurrence(q[None, :, None], k[None, :, None], v[None, :, None],
                              g[None, :, None], beta[None, :, None], S0[None, None])
    F = lambda a: [[Fr(float(x)) for x in row] for row in a]
    outs, Sf = _frac_matrix_recurrence(F(S0), F(k), F(v), F(q),
                                       [Fr(float(b)) for b in beta],
                                       [Fr(float(a)) for a in alpha_fp])
    ref_o = np.array([[float(x) for x in row] for row in outs])
    ref_S = np.array([[float(x) for x in row] for row in Sf])
    np.testing.assert_allclose(o[0, :, 0], ref_o, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(ST[0, 0], ref_S, rtol=1e-13, atol=1e-13)


# --------------------------------------------------------------------------- limits
def test_beta_zero_is_pure_decay():
    q, k, v, g, beta, S0 = _rand(11, T=17)
    beta[:] = 0.0
    o, ST = oracle.recurrence(q, k, v, g, beta, S0)
    G = np.cumsum(g, axis=1)                                     # [B,T,H]
    for h in range(q.shape[2]):
        np.testing.assert_allclose(ST[0, h], math.exp(G[0, -1, h]) * S0[0, h], rtol=1e-12)
        ref_o = np.exp(G[0, :, h])[:, None] * (q[0, :, h] @ S0[0, h].T)
        np.testing.assert_allclose(o[0, :, h], ref_o, rtol=1e-12, atol=1e-15)


def test_alpha_one_beta_one_orthonormal_keys_write_columns():
    """alpha=1: plain delta rule; unit keys e_t with beta=1 store v_t in column t."""
    dk, dv, T, H = 8, 5, 6, 1
    rng = np.random.default_rng(5)
    k = np.zeros((1, T, H, dk))
    for t in range(T):
        k[0, t, 0, t] = 1.0
    q = rng.standard_normal((1, T, H, dk))
    v = rng.standard_normal((1, T, H, dv))
    g = np.zeros((1, T, H))
    beta = np.ones((1, T, H))
    S0 = rng.standard_normal((1, H, dv, dk))
    o, ST = oracle.recurrence(q, k, v, g, beta, S0)
    expect = S0[0, 0].copy()
    expect[:, :T] = v[0, :, 0].T            # S0 (I - sum e e^T) + sum v e^T
    np.testing.assert_array_equal(ST[0, 0], expect)
    # the readout after token t sees columns 0..t overwritten
    for t in range(T):
        St = S0[0, 0].copy()
        St[:, :t + 1] = v[0, :t + 1, 0].T
        np.testing.assert_allclose(o[0, t, 0], St @ q[0, t, 0], rtol=1e-14, atol=1e-14)


def test_alpha_one_matches_lms_update():
    """At alpha = 1 the rule is the Widrow-Hoff LMS step S <- S + beta (v - S k) k^T."""
    q, k, v, g, beta, S0 = _rand(21, T=9, H=1)
    g[:] = 0.0
    o, ST = oracle.recurrence(q, k, v, g, beta, S0)
    S = S0[0, 0].copy()
    for t in range(q.shape[1]):
        kt, vt = k[0, t, 0], v[0, t, 0]
        err = vt - S @ kt
        S = S + beta[0, t, 0] * np.outer(err, kt)
        np.testing.assert_allclose(o[0, t, 0], S @ q[0, t, 0], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(ST[0, 0], S, rtol=1e-12, atol=1e-14)


def test_alpha_to_zero_forgets_everything():
    """g = -1e4 underflows alpha to 0: S_t = beta_t v_t k_t^T, o_t = beta_t (k_t.q_t) v_t."""
    q, k, v, g, beta, S0 = _rand(31, T=7)
    g[:] = -1e4
    o, ST = oracle.recurrence(q, k, v, g, beta, S0)
    kq = np.sum(k * q, axis=-1)
    np.testing.assert_allclose(o, (beta * kq)[..., None] * v, rtol=1e-13, atol=1e-15)
    for h in range(q.shape[2]):
        np.testing.assert_allclose(ST[0, h], beta[0, -1, h] * np.outer(v[0, -1, h], k[0, -1, h]),
                                   rtol=1e-13, atol=1e-15)


# --------------------------------------------------------------------------- invariants
def test_linear_in_values_and_initial_state():
    q, k, v1, g, beta, S1 = _rand(41, T=15)
    _, _, v2, _, _, S2 = _rand(42, T=15)
    a, b = 0.75, -1.25
    o1, T1 = oracle.recurrence(q, k, v1, g, beta, S1)
    o2, T2 = oracle.recurrence(q, k, v2, g, beta, S2)
    o3, T3 = oracle.recurrence(q, k, a * v1 + b * v2, g, beta, a * S1 + b * S2)
    np.testing.assert_allclose(o3, a * o1 + b * o2, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(T3, a * T1 + b * T2, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("split", [1, 5, 12])
def test_state_passing_split_equals_whole(split):
    q, k, v, g, beta, S0 = _rand(51, T=13)
    o, ST = oracle.recurrence(q, k, v, g, beta, S0)
    sl = lambda x, a, b: x[:, a:b]
    oa, Sa = oracle.recurrence(*(sl(x, 0, split) for x in (q, k, v, g, beta)), S0)
    ob, Sb = oracle.recurrence(*(sl(x, split, None) for x in (q, k, v, g, beta)), Sa)
    np.testing.assert_allclose(np.concatenate([oa, ob], axis=1), o, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(Sb, ST, rtol=1e-13, atol=1e-14)


def test_decode_steps_equal_prefill():
    q, k, v, g, beta, S0 = _rand(61, T=6, B=2)
    o, ST = oracle.recurrence(q, k, v, g, beta, S0)
    S = S0.copy()
    for t in range(q.shape[1]):
        ot, S = oracle.decode_step(q[:, t], k[:, t], v[:, t], g[:, t], beta[:, t], S)
        np.testing.assert_allclose(ot, o[:, t], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(S, ST, rtol=1e-13, atol=1e-14)


def test_heads_are_independent_and_equivariant():
    q, k, v, g, beta, S0 = _rand(71, T=9, H=4)
    perm = np.array([2, 0, 3, 1])
    o, ST = oracle.recurrence(q, k, v, g, beta, S0)
    op, STp = oracle.recurrence(q[:, :, perm], k[:, :, perm], v[:, :, perm], g[:, :, perm],
                                beta[:, :, perm], S0[:, perm])
    np.testing.assert_array_equal(op, o[:, :, perm])
    np.testing.assert_array_equal(STp, ST[:, perm])


def test_ragged_packing_equals_separate_calls():
    lens = [5, 0, 11, 1]
    cu = np.concatenate([[0], np.cumsum(lens)])
    q, k, v, g, beta, _ = _rand(81, T=int(cu[-1]), H=2)
    S0 = np.random.default_rng(82).standard_normal((len(lens), 2, 3, 5))
    o, ST = oracle.recurrence(q, k, v, g, beta, S0, cu_seqlens=cu)
    for s in range(len(lens)):
        a, b = cu[s], cu[s + 1]
        os_, Ss = oracle.recurrence(*(x[:, a:b] for x in (q, k, v, g, beta)), S0[s:s + 1])
        np.testing.assert_array_equal(o[:, a:b], os_)
        np.testing.assert_array_equal(ST[s], Ss[0])
    np.testing.assert_array_equal(ST[1], S0[1])           # empty sequence keeps its state


def test_spectral_norm_bound():
    """||S_t||_2 <= alpha_t ||S_{t-1}||_2 + beta_t ||v_t|| for unit keys, beta in [0,1]."""
    q, k, v, g, beta, S0 = _rand(91, T=12, H=1)
    S_prev = S0[0, 0]
    for t in range(q.shape[1]):
        _, S = oracle.recurrence(*(x[:, t:t + 1] for x in (q, k, v, g, beta)), S_prev[None, None])
        lhs = np.linalg.norm(S[0, 0], 2)
        rhs = math.exp(g[0, t, 0]) * np.linalg.norm(S_prev, 2) + beta[0, t, 0] * np.linalg.norm(v[0, t, 0])
        assert lhs <= rhs * (1 + 1e-12)
        S_prev = S[0, 0]


def test_retrieval_identity_per_step():
    """Reading with q_t = k_t (unit) gives alpha_t (1 - beta_t) S_{t-1} k_t + beta_t v_t."""
    q, k, v, g, beta, S0 = _rand(95, T=10, H=1)
    q = k.copy()
    o, _ = oracle.recurrence(q, k, v, g, beta, S0)
    S_prev = S0[0, 0]
    for t in range(q.shape[1]):
        a, b = math.exp(g[0, t, 0]), beta[0, t, 0]
        expect = a * (1 - b) * (S_prev @ k[0, t, 0]) + b * v[0, t, 0]
        np.testing.assert_allclose(o[0, t, 0], expect, rtol=1e-12, atol=1e-14)
        _, S = oracle.recurrence(*(x[:, t:t + 1] for x in (q, k, v, g, beta)), S_prev[None, None])
        S_prev = S[0, 0]


def test_scale_multiplies_output_only():
    q, k, v, g, beta, S0 = _rand(97, T=8)
    o1, S1 = oracle.recurrence(q, k, v, g, beta, S0)
    o2, S2 = oracle.recurrence(q, k, v, g, beta, S0, scale=0.125)
    np.testing.assert_allclose(o2, 0.125 * o1, rtol=1e-14, atol=1e-16)
    np.testing.assert_array_equal(S1, S2)


# --------------------------------------------------------------------------- chunked form
@pytest.mark.parametrize("chunk", list(range(1, 70)))
def test_chunked_equals_sequential_every_chunk_size(chunk):
    q, k, v, g, beta, S0 = _rand(101, T=67, H=1, dk=6, dv=4)
    o, ST = oracle.recurrence(q, k, v, g, beta, S0)
    oc, STc = ch.chunked(q, k, v, g, beta, S0, chunk=chunk)
    np.testing.assert_allclose(oc, o, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(STc, ST, rtol=1e-11, atol=1e-12)


def test_chunked_ragged_and_fast_decay():
    lens = [70, 3, 128, 64]
    cu = np.concatenate([[0], np.cumsum(lens)])
    q, k, v, g, beta, _ = _rand(103, T=int(cu[-1]), H=2, dk=8, dv=8, g_scale=3.0)
    g -= 2.0                                                   # per-chunk sum of g far below -88
    S0 = np.random.default_rng(104).standard_normal((len(lens), 2, 8, 8))
    o, ST = oracle.recurrence(q, k, v, g, beta, S0, cu_seqlens=cu)
    oc, STc = ch.chunked(q, k, v, g, beta, S0, chunk=64, cu_seqlens=cu)
    np.testing.assert_allclose(oc, o, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(STc, ST, rtol=1e-10, atol=1e-12)


def test_chunk_terms_solve_their_triangular_systems():
    q, k, v, g, beta, _ = _rand(105, T=64, H=1, dk=16, dv=8)
    tm = ch.chunk_terms(q[0, :, 0], k[0, :, 0], v[0, :, 0], g[0, :, 0], beta[0, :, 0])
    n = 64
    I = np.eye(n)
    np.testing.assert_allclose(tm["T"] @ (I + tm["A"]), I, atol=1e-12)
    assert np.all(np.triu(tm["A"]) == 0)
    assert np.all(np.triu(tm["P"], 1) == 0)
    gam = np.exp(np.cumsum(g[0, :, 0]))
    np.testing.assert_allclose((I + tm["A"]) @ tm["W"], (beta[0, :, 0] * gam)[:, None] * k[0, :, 0],
                               atol=1e-12)


# --------------------------------------------------------------------------- grouped key heads
def _grouped_brute(q, k, v, g, beta, S0, G):
    """Per value head h, token by token, with the rank-1 form and the key head h // G chosen by hand."""
    B, T, H, dv = v.shape
    dk = q.shape[-1]
    o = np.zeros((B, T, H, dv))
    ST = np.zeros((B, H, dv, dk))
    for b in range(B):
        for h in range(H):
            kh = h // G
            S = np.zeros((dv, dk)) if S0 is None else S0[b, h].copy()
            for t in range(T):
                kt, qt = k[b, t, kh], q[b, t, kh]
                a, bt = math.exp(g[b, t, h]), beta[b, t, h]
                S = a * (S - bt * np.outer(S @ kt, kt)) + bt * np.outer(v[b, t, h], kt)
                o[b, t, h] = S @ qt
            ST[b, h] = S
    return o, ST


@pytest.mark.parametrize("H,Hk", [(4, 2), (6, 3), (4, 1), (3, 3)])
def test_grouped_key_heads_brute_force(H, Hk):
    """Value head h reads key head h // (H / H_k): checked against a hand loop over heads."""
    rng = np.random.default_rng(40 + H * 7 + Hk)
    B, T, dk, dv = 2, 9, 4, 3
    q = rng.standard_normal((B, T, Hk, dk))
    k = rng.standard_normal((B, T, Hk, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, T, H, dv))
    beta = 1 / (1 + np.exp(-rng.standard_normal((B, T, H))))
    g = -np.logaddexp(0, rng.standard_normal((B, T, H)))
    S0 = 0.3 * rng.standard_normal((B, H, dv, dk))
    o, ST = oracle.recurrence_grouped(q, k, v, g, beta, S0)
    ro, rS = _grouped_brute(q, k, v, g, beta, S0, H // Hk)
    np.testing.assert_allclose(o, ro, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(ST, rS, rtol=1e-12, atol=1e-12)


def test_grouped_heads_sharing_a_key_head_differ_only_through_their_own_inputs():
    """Two value heads of one group with equal v, g, beta give equal results; a head of another group does not."""
    rng = np.random.default_rng(77)
    B, T, H, Hk, dk, dv = 1, 11, 4, 2, 5, 3
    q = rng.standard_normal((B, T, Hk, dk))
    k = rng.standard_normal((B, T, Hk, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = np.repeat(rng.standard_normal((B, T, 1, dv)), H, axis=2)
    beta = np.full((B, T, H), 0.6)
    g = np.full((B, T, H), -0.2)
    o, ST = oracle.recurrence_grouped(q, k, v, g, beta)
    np.testing.assert_array_equal(o[:, :, 0], o[:, :, 1])
    np.testing.assert_array_equal(o[:, :, 2], o[:, :, 3])
    assert np.abs(o[:, :, 0] - o[:, :, 2]).max() > 1e-3


def test_grouped_decode_equals_grouped_prefill():
    rng = np.random.default_rng(78)
    B, T, H, Hk, dk, dv = 2, 6, 4, 2, 5, 3
    q = rng.standard_normal((B, T, Hk, dk))
    k = rng.standard_normal((B, T, Hk, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((B, T, H, dv))
    beta = 1 / (1 + np.exp(-rng.standard_normal((B, T, H))))
    g = -np.logaddexp(0, rng.standard_normal((B, T, H)))
    S = 0.1 * rng.standard_normal((B, H, dv, dk))
    o, ST = oracle.recurrence_grouped(q, k, v, g, beta, S)
    for t in range(T):
        ot, S = oracle.decode_step_grouped(q[:, t], k[:, t], v[:, t], g[:, t], beta[:, t], S)
        np.testing.assert_allclose(ot, o[:, t], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(S, ST, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------- in-kernel input transforms
def test_gate_logits_closed_forms():
    """a = 0 gives alpha = 1/2 exactly; b = 0 gives beta = 1/2; softplus against math.log1p(math.exp(a))."""
    a = np.array([0.0, -3.5, 2.25, 10.0, -30.0])
    b = np.array([0.0, 1.0, -2.0, 4.0, -8.0])
    g, beta = oracle.gates_from_logits(a, b)
    for ai, gi in zip(a, g):
        assert abs(gi + math.log1p(math.exp(ai))) < 1e-14 * max(1.0, abs(ai))
    for bi, be in zip(b, beta):
        assert abs(be - 1.0 / (1.0 + math.exp(-bi))) < 1e-15
    assert abs(math.exp(g[0]) - 0.5) < 1e-15 and beta[0] == 0.5
    # through the recurrence: logits (0, 0) everywhere = alpha = beta = 1/2 given directly
    q, k, v, _, _, S0 = _rand(51, T=9)
    z = np.zeros(q.shape[:3])
    o1, s1 = oracle.recurrence_ex(q, k, v, z, z, S0, gate_logits=True)
    o2, s2 = oracle.recurrence(q, k, v, z - math.log(2.0), z + 0.5, S0)
    np.testing.assert_allclose(o1, o2, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(s1, s2, rtol=1e-13, atol=1e-14)


def test_l2_transform_against_hand_normalised_rows_and_scale_invariance():
    rng = np.random.default_rng(52)
    B, T, H, dk, dv = 1, 10, 2, 6, 3
    q = 3.0 * rng.standard_normal((B, T, H, dk))
    k = 0.5 * rng.standard_normal((B, T, H, dk))
    v = rng.standard_normal((B, T, H, dv))
    g = -np.logaddexp(0, rng.standard_normal((B, T, H)))
    beta = 1 / (1 + np.exp(-rng.standard_normal((B, T, H))))

    def unit(x):   # row by row with math.sqrt
        y = np.empty_like(x)
        for idx in np.ndindex(x.shape[:-1]):
            y[idx] = x[idx] / math.sqrt(sum(float(t) * float(t) for t in x[idx]) + 1e-6)
        return y
    o1, s1 = oracle.recurrence_ex(q, k, v, g, beta, qk_l2norm=True)
    o2, s2 = oracle.recurrence(unit(q), unit(k), v, g, beta)
    np.testing.assert_allclose(o1, o2, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(s1, s2, rtol=1e-12, atol=1e-13)
    # a positive factor per (token, head) on q or k changes nothing beyond the epsilon's share
    c = np.exp(rng.uniform(-1, 1, size=(B, T, H, 1)))
    # (rows here have |x|^2 > 0.09, so the epsilon moves each by under 6e-6 relative)
    o3, s3 = oracle.recurrence_ex(q * c, k / c, v, g, beta, qk_l2norm=True)
    np.testing.assert_allclose(o3, o1, rtol=0, atol=1e-4 * np.abs(o1).max())
    np.testing.assert_allclose(s3, s1, rtol=0, atol=1e-4 * np.abs(s1).max())
    # a zero key row writes nothing: that token only decays the state
    k0 = k.copy()
    k0[0, 4, 1] = 0.0
    _, sa = oracle.recurrence_ex(q[:, :5], k0[:, :5], v[:, :5], g[:, :5], beta[:, :5], qk_l2norm=True)
    _, sb = oracle.recurrence_ex(q[:, :4], k0[:, :4], v[:, :4], g[:, :4], beta[:, :4], qk_l2norm=True)
    np.testing.assert_allclose(sa[0, 1], math.exp(g[0, 4, 1]) * sb[0, 1], rtol=1e-13, atol=1e-15)


def test_ex_decode_equals_ex_prefill():
    rng = np.random.default_rng(53)
    B, T, H, Hk, dk, dv = 2, 5, 4, 2, 5, 3
    q = 2.0 * rng.standard_normal((B, T, Hk, dk))
    k = rng.standard_normal((B, T, Hk, dk))
    v = rng.standard_normal((B, T, H, dv))
    a = rng.standard_normal((B, T, H))
    b = rng.standard_normal((B, T, H))
    S = 0.1 * rng.standard_normal((B, H, dv, dk))
    kw = dict(qk_l2norm=True, gate_logits=True)
    o, ST = oracle.recurrence_ex(q, k, v, a, b, S, **kw)
    for t in range(T):
        ot, S = oracle.decode_step_ex(q[:, t], k[:, t], v[:, t], a[:, t], b[:, t], S, **kw)
        np.testing.assert_allclose(ot, o[:, t], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(S, ST, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------- causal attention oracle
from oracle import attention as att  # noqa: E402


def _att_brute(q, k, v, scale):
    """Pure-Python loops with math.exp: o_i = sum_{j<=i} e^{s_ij} v_j / sum_{j<=i} e^{s_ij}."""
    B, T, H, d = q.shape
    Hkv = k.shape[2]
    o = np.zeros(q.shape)
    for b in range(B):
        for h in range(H):
            kh = h // (H // Hkv)
            for i in range(T):
                s = [scale * sum(float(q[b, i, h, c]) * float(k[b, j, kh, c]) for c in range(d)) for j in range(i + 1)]
                mx = max(s)
                w = [math.exp(x - mx) for x in s]
                z = sum(w)
                for c in range(d):
                    o[b, i, h, c] = sum(w[j] * float(v[b, j, kh, c]) for j in range(i + 1)) / z
    return o


@pytest.mark.parametrize("H,Hkv", [(2, 1), (4, 2), (3, 3)])
def test_attention_brute_force(H, Hkv):
    rng = np.random.default_rng(60 + H + Hkv)
    q = rng.standard_normal((2, 7, H, 3))
    k = rng.standard_normal((2, 7, Hkv, 3))
    v = rng.standard_normal((2, 7, Hkv, 3))
    np.testing.assert_allclose(att.causal_attention(q, k, v, 0.7), _att_brute(q, k, v, 0.7), rtol=1e-12, atol=1e-13)


def test_attention_closed_forms():
    rng = np.random.default_rng(61)
    B, T, H, d = 1, 9, 2, 4
    q = rng.standard_normal((B, T, H, d))
    k = np.repeat(rng.standard_normal((B, 1, 1, d)), T, axis=1)   # one key everywhere
    v = rng.standard_normal((B, T, 1, d))
    o = att.causal_attention(q, k, v, 0.5)
    prefix_mean = np.cumsum(v[:, :, 0], axis=1) / np.arange(1, T + 1)[None, :, None]
    for h in range(H):
        np.testing.assert_allclose(o[:, :, h], prefix_mean, rtol=1e-13, atol=1e-14)   # equal scores: prefix means
    k2 = rng.standard_normal((B, T, 1, d))
    o2 = att.causal_attention(q, k2, v, 0.0)                                          # scale 0: the same
    np.testing.assert_allclose(o2[:, :, 0], prefix_mean, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(o2[:, 0, 1], v[:, 0, 0], rtol=0, atol=0)               # first query sees only key 0


def test_attention_invariances_and_sampled_rows():
    rng = np.random.default_rng(62)
    B, T, H, Hkv, d = 2, 40, 4, 2, 8
    q = rng.standard_normal((B, T, H, d))
    k = rng.standard_normal((B, T, Hkv, d))
    v = rng.standard_normal((B, T, Hkv, d))
    o = att.causal_attention(q, k, v, 0.35)
    u = rng.standard_normal(d)            # k_j + u adds q_i.u to every score of row i: softmax unchanged
    np.testing.assert_allclose(att.causal_attention(q, k + u, v, 0.35), o, rtol=1e-10, atol=1e-12)
    rows = [0, 5, 17, 39]
    np.testing.assert_allclose(att.causal_attention(q, k, v, 0.35, rows=rows), o[:, rows], rtol=1e-13, atol=1e-14)
    # a value change at position j reaches only queries i >= j
    v2 = v.copy()
    v2[:, 20] += 1.0
    o2 = att.causal_attention(q, k, v2, 0.35)
    assert np.array_equal(o2[:, :20], o[:, :20]) and np.abs(o2[:, 20:] - o[:, 20:]).min() > 0
