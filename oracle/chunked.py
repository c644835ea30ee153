"""Chunked (intra-/inter-chunk) form of the gated delta rule, fp64 numpy.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The steps run in the order of the chunked scan of section 3.2, in the paper's
state orientation S_p in R^{dk x dv} (the transpose of the [dv, dk] storage
used everywhere else).  Per chunk of n tokens: the key-key and query-key
products; the unit-lower-triangular solve by forward substitution, which needs
nothing from the state entering the chunk; the products that form the
correction and the outputs.  Then, once every chunk's (M_c, N_c) exists, the
inter-chunk step S_p <- M_c S_p + N_c walks the chunks in order.

Derivation (per state column, i.e. per value channel): with
G_r = sum_{j<=r} g_j, gamma_r = exp(G_r) and Gamma_{ri} = exp(G_r - G_i) for i <= r,
unrolling S_r = alpha_r S_{r-1} + k_r u_r^T inside the chunk gives

    (I + A) U = diag(beta) V - diag(beta*gamma) K S_p0,
    A_ri      = beta_r Gamma_ri (k_r . k_i)           (i < r, else 0)
    O         = diag(gamma) Q S_p0 + (Q K^T o Gamma)_{i<=r} U
    S_pn      = gamma_n S_p0 + K^T diag(exp(G_n - G_r)) U,

so with T = (I + A)^{-1}, W = T diag(beta gamma) K and Ut = T diag(beta) V:
U = Ut - W S_p0, M_c = gamma_n I - K^T D W and N_c = K^T D Ut.
Pure-python loops only over chunks and over the rows of the triangular solve.
"""
from __future__ import annotations

import numpy as np


def forward_substitution(A, rhs):
    """Solve (I + A) X = rhs for strictly lower-triangular A, row by row."""
    n = A.shape[0]
    X = np.zeros_like(rhs)
    for r in range(n):
        X[r] = rhs[r] - A[r, :r] @ X[:r]
    return X


def chunk_terms(q, k, v, g, beta, scale=1.0):
    """State-independent quantities of one chunk (n tokens, one head).

    q,k [n,dk]; v [n,dv]; g,beta [n].  Returns a dict with G, A, T, P, W, Ut,
    M, N (paper orientation).
    """
    q = np.asarray(q, np.float64) * scale
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    g = np.asarray(g, np.float64)
    beta = np.asarray(beta, np.float64)
    n, dk = k.shape
    G = np.cumsum(g)
    gamma = np.exp(G)
    lower = np.tril(np.ones((n, n), dtype=bool))
    diff = np.where(lower, G[:, None] - G[None, :], -np.inf)   # mask before exp
    Gam = np.exp(diff)
    KK = k @ k.T                                   # token-token products
    QK = q @ k.T
    A = np.tril(beta[:, None] * KK * Gam, -1)
    P = QK * Gam                                   # zero above the diagonal
    # forward substitution, right-hand sides independent of the incoming state
    W = forward_substitution(A, (beta * gamma)[:, None] * k)
    Ut = forward_substitution(A, beta[:, None] * v)
    T = forward_substitution(A, np.eye(n))
    D = np.exp(G[-1] - G)
    M = gamma[-1] * np.eye(dk) - k.T @ (D[:, None] * W)
    N = k.T @ (D[:, None] * Ut)
    return dict(G=G, gamma=gamma, A=A, T=T, P=P, W=W, Ut=Ut, M=M, N=N, q=q)


def chunked(q, k, v, g, beta, S0=None, *, chunk=64, cu_seqlens=None, scale=1.0):
    """Same contract as :func:`oracle.recurrence`, computed chunk-wise."""
    q, k, v, g, beta = (np.asarray(x, np.float64) for x in (q, k, v, g, beta))
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    if cu_seqlens is None:
        seqs = [(b, 0, T) for b in range(B)]
    else:
        cu = [int(x) for x in cu_seqlens]
        seqs = [(0, cu[s], cu[s + 1]) for s in range(len(cu) - 1)]
    o = np.zeros((B, T, H, dv))
    ST = np.zeros((len(seqs), H, dv, dk))
    for s, (b, t0, t1) in enumerate(seqs):
        for h in range(H):
            Sp = np.zeros((dk, dv)) if S0 is None else np.asarray(S0, np.float64)[s, h].T.copy()
            starts = list(range(t0, t1, chunk))
            # every (M_c, N_c) and every chunk's local terms before the recurrence
            terms = [chunk_terms(q[b, c0:min(c0 + chunk, t1), h], k[b, c0:min(c0 + chunk, t1), h],
                                 v[b, c0:min(c0 + chunk, t1), h], g[b, c0:min(c0 + chunk, t1), h],
                                 beta[b, c0:min(c0 + chunk, t1), h], scale)
                     for c0 in starts]
            for c0, tm in zip(starts, terms):
                n = len(tm["G"])
                U = tm["Ut"] - tm["W"] @ Sp                       # per-chunk correction
                o[b, c0:c0 + n, h] = tm["gamma"][:, None] * (tm["q"] @ Sp) + tm["P"] @ U
                Sp = tm["M"] @ Sp + tm["N"]                       # inter-chunk recurrence
            ST[s, h] = Sp.T
    return o, ST
