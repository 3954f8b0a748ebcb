"""Chunked (WY / UT) form of the gated delta rule in fp64 -- TEST INFRASTRUCTURE ONLY.

This is an independent algebraic rewrite of the token recurrence, used only to
pin the recurrence in ``gdn_oracle.c`` (and never for GPU parity).  It is the
token-wise analog of the paper's split of the update into per-frame summaries
followed by a short sequential scan (Section "Efficient System Co-design",
paragraph "Efficient GDN Kernel": ``S_f = alpha_f P_f S_{f-1} + A_f``).

Derivation (state stored as H = S^T, shape [Dk, Dv]).  Write one token step as
``H_r = alpha_r H_{r-1} + k_r u_r^T`` with the pseudo-value
``u_r = beta_r (v_r - alpha_r H_{r-1}^T k_r)`` (decay, then write the residual:
equation appendix_gdn_kv_update with one token).  Inside a chunk with entry
state H_0 let ``G[r, s] = prod_{s < u <= r} alpha_u`` (G[r, r] = 1) and
``gam_r = prod_{u <= r} alpha_u``.  Unrolling gives
``H_r = gam_r H_0 + sum_{s <= r} G[r, s] k_s u_s^T``; substituting into u_r:

    u_r + sum_{s < r} beta_r G[r, s] (k_r . k_s) u_s = beta_r v_r - beta_r gam_r H_0^T k_r

so with ``A[r, s] = beta_r G[r, s] (k_r . k_s)`` (s < r), ``T = (I + A)^-1``:

    U = Ut - W H_0,   Ut = T diag(beta) V,   W = T diag(beta * gam) K
    O = diag(gam) Q H_0 + (Q K^T o M) U,     M[r, s] = G[r, s] for s <= r else 0
    H_C = gam_C H_0 + K^T diag(G[C, :]) U

The decay products are formed directly from alpha (no logarithms), so
alpha = 0 is exact.  The triangular solve uses scipy's solver as a primitive.
"""
import numpy as np
from scipy.linalg import solve_triangular


def _f64(x):
    x = np.asarray(x)
    if x.dtype == np.uint16:  # bf16 bit patterns, widened exactly
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def _decay_matrix(a):
    """G[r, s] = prod_{s < u <= r} a_u for s <= r, else 0 (brute force)."""
    n = a.shape[0]
    G = np.zeros((n, n))
    for s in range(n):
        G[s, s] = 1.0
        for r in range(s + 1, n):
            G[r, s] = G[r - 1, s] * a[r]
    return G


def chunk_step(Q, K, V, a, b, H0):
    """One chunk: Q, K [n, Dk]; V [n, Dv]; a, b [n]; H0 [Dk, Dv] -> (O [n, Dv], H_C)."""
    n = K.shape[0]
    G = _decay_matrix(a)
    gam = np.cumprod(a)                       # gam_r = prod_{u <= r} a_u
    A = np.tril(b[:, None] * G * (K @ K.T), k=-1)
    I = np.eye(n)
    T = solve_triangular(I + A, I, lower=True, unit_diagonal=True)
    W = T @ ((b * gam)[:, None] * K)
    Ut = T @ (b[:, None] * V)
    U = Ut - W @ H0
    M = np.tril(G)
    O = gam[:, None] * (Q @ H0) + (np.tril(Q @ K.T) * M) @ U
    HC = gam[-1] * H0 + K.T @ (G[-1, :][:, None] * U)
    return O, HC


def gdn_chunked(q, k, v, alpha, beta, state_in=None, chunk=64):
    """Chunked evaluation over [B, T, H, D] inputs; returns (out, state_out) in fp64."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    alpha, beta = _f64(alpha), _f64(beta)
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    out = np.zeros((B, T, H, Dv))
    state = np.zeros((B, H, Dk, Dv))
    for b in range(B):
        for h in range(H):
            Hs = np.zeros((Dk, Dv)) if state_in is None else _f64(state_in[b, h]).copy()
            for c0 in range(0, T, chunk):
                sl = slice(c0, min(c0 + chunk, T))
                O, Hs = chunk_step(q[b, sl, h], k[b, sl, h], v[b, sl, h],
                                   alpha[b, sl, h], beta[b, sl, h], Hs)
                out[b, sl, h] = O
            state[b, h] = Hs
    return out, state
