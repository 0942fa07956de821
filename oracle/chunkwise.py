"""Chunkwise-parallel algebra of App. D in float64.  TEST INFRASTRUCTURE ONLY
(see the package header).

The token recurrence in `recurrent` is the definition; the functions here
restate the paper's chunkwise forms literally (dense C x C matrices, a
library triangular solve, no blocking or fusion) so that (a) the tests can
check that the two agree to rounding, and (b) the GPU tests can compare each
kernel's intermediate (write key, T, W, U, E, chunk-start states) with the
quantity the paper defines.

Orientation and layout as in `recurrent`: S is (N, dv, dk) in the paper's
orientation; per-token tensors are (N, T, d).  A chunk is C consecutive
tokens; the last chunk may be shorter (ragged tail).
"""
from __future__ import annotations

import numpy as np

from .recurrent import squash, _f64


def chunk_bounds(T, C):
    return [(s, min(s + C, T)) for s in range(0, T, C)]


def gram_chunkwise(k, beta_p, g_p, C, A0=None):
    """Chunkwise form of the decayed diagonal-Gram recurrence
    A_t = alpha^P_t A_{t-1} + beta^P_t k_t^2 (App. D, "Chunkwise parallel
    forms for the preconditioner recurrences", Eq. precond_from_boundary):

    within chunk i with boundary state A_b,
        A_[i]   = Phi_left 1 A_b^T + M_[i] Diag(beta^P) K^(2)
        A_end   = (prod alpha) A_b + 1^T Phi_right Diag(beta^P) K^(2)
    where M_[i][j,l] = prod_{l<m<=j} alpha_m (j >= l), Phi_left_jj =
    prod_{m<=j} alpha_m and Phi_right_jj = prod_{m>j} alpha_m.

    Returns (A_all (N,T,dk) with A_all[:, t] = A_t, A_bound (N, NT+1, dk))
    where A_bound[:, i] is the state before chunk i."""
    k = _f64(k)
    N, T, dk = k.shape
    beta_p = _f64(beta_p)
    gp = np.zeros((N, T)) if g_p is None else _f64(g_p)
    A_b = np.zeros((N, dk)) if A0 is None else _f64(A0).copy()
    A_all = np.empty_like(k)
    bounds = chunk_bounds(T, C)
    A_bound = np.empty((N, len(bounds) + 1, dk))
    for i, (s, e) in enumerate(bounds):
        A_bound[:, i] = A_b
        K2 = k[:, s:e] ** 2                                  # K^(2)
        lp = np.cumsum(gp[:, s:e], axis=1)                   # log prod_{m<=j}
        n = e - s
        diff = lp[:, :, None] - lp[:, None, :]               # log prod_{l<m<=j}
        with np.errstate(over="ignore"):
            M = np.where(np.tril(np.ones((n, n), bool))[None], np.exp(diff),
                         0.0)
        bK2 = beta_p[:, s:e, None] * K2
        A_all[:, s:e] = np.exp(lp)[:, :, None] * A_b[:, None, :] + M @ bK2
        phi_right = np.exp(lp[:, -1:] - lp)                  # prod_{m>j}
        A_b = np.exp(lp[:, -1])[:, None] * A_b + np.einsum(
            "nj,njd->nd", phi_right, bK2)
    A_bound[:, len(bounds)] = A_b
    return A_all, A_bound


def preconditioner_chunkwise(k, beta_p, g_p, mu, x, C, A0=None):
    """Stable ATK write key from the chunkwise Gram states (App. D, "ATK
    (stable) preconditioner recurrence": no left shift, then B = F(A),
    Kt = B * K), with A_t from `gram_chunkwise`.

    Returns (kt (N,T,dk), A_bound (N, NT+1, dk)) where A_bound[:, i] is the
    state before chunk i."""
    k = _f64(k)
    N = k.shape[0]
    A_all, A_bound = gram_chunkwise(k, beta_p, g_p, C, A0)
    kt = squash(A_all, _f64(mu).reshape(N, 1, 1), x) * k
    return kt, A_bound


def _decay_factors(g, gate, N, s, e, dk):
    """Lambda_r = exp(G_r) with G the inclusive in-chunk prefix of the
    log-decay (gamma_r of App. D for the scalar gate; Lambda of the KDA form
    for the per-channel gate).  Returned as (N, n, dk)."""
    n = e - s
    if gate == "none":
        return np.ones((N, n, dk))
    G = np.cumsum(_f64(g)[:, s:e], axis=1)
    if gate == "scalar":
        return np.repeat(np.exp(G)[:, :, None], dk, axis=2)
    return np.exp(G)


def chunk_forward(q, k, kt, v, beta, g=None, gate="none", S0=None, C=64,
                  scale=1.0, keep=False):
    """Chunkwise PDN / PGDN / PKDA forward (Eq. chunkwise_atk_form; App. D
    "PDN chunkwise parallel form", "Scalar-decayed PDN", "Diagonally-decayed
    PDN").  Per chunk, with Lambda from `_decay_factors`:

        At  = tril(Diag(beta) (K*Lam)(Kt/Lam)^T, -1)
        Tm  = (I + At)^{-1} Diag(beta)                    (Eq. T_two_key)
        W   = Tm (Lam*K),   U = Tm V                      (Eq. WU_two_key)
        E   = U - W S^T
        O   = scale [ (Q*Lam) S^T + tril((Q*Lam)(Kt/Lam)^T) E ]
        S  <- S Diag(Lam_C) + E^T (Kt * Lam_C/Lam)

    The gated W, U and At are our reading of the decayed forms, which the
    paper states without their UT system.  Returns (o, S_T) or, with
    keep=True, (o, S_T, inter) where inter holds per-token W, U, E (N,T,.),
    Tm (N,NT,C,C) and the chunk-start states S_start (N,NT,dv,dk)."""
    q, k, kt, v, beta = map(_f64, (q, k, kt, v, beta))
    N, T, dk = k.shape
    dv = v.shape[2]
    S = np.zeros((N, dv, dk)) if S0 is None else _f64(S0).copy()
    o = np.empty((N, T, dv))
    bounds = chunk_bounds(T, C)
    if keep:
        W_all = np.empty((N, T, dk))
        U_all = np.empty((N, T, dv))
        E_all = np.empty((N, T, dv))
        T_all = np.zeros((N, len(bounds), C, C))
        S_start = np.empty((N, len(bounds), dv, dk))
    for i, (s, e) in enumerate(bounds):
        n = e - s
        Lam = _decay_factors(g, gate, N, s, e, dk)
        Q, K, Kt, V = q[:, s:e], k[:, s:e], kt[:, s:e], v[:, s:e]
        b = beta[:, s:e]
        strict = np.tril(np.ones((n, n), bool), -1)
        causal = np.tril(np.ones((n, n), bool))
        At = np.where(strict, b[:, :, None] * ((K * Lam) @ np.swapaxes(
            Kt / Lam, 1, 2)), 0.0)
        Tm = np.linalg.solve(np.eye(n)[None] + At,
                             np.eye(n)[None] * b[:, None, :])
        W = Tm @ (Lam * K)
        U = Tm @ V
        E = U - W @ np.swapaxes(S, 1, 2)
        P = np.where(causal, (Q * Lam) @ np.swapaxes(Kt / Lam, 1, 2), 0.0)
        o[:, s:e] = scale * ((Q * Lam) @ np.swapaxes(S, 1, 2) + P @ E)
        if keep:
            W_all[:, s:e], U_all[:, s:e], E_all[:, s:e] = W, U, E
            T_all[:, i, :n, :n] = Tm
            S_start[:, i] = S
        LamC = Lam[:, -1:, :]
        S = S * LamC + np.swapaxes(E, 1, 2) @ (Kt * (LamC / Lam))
    if keep:
        return o, S, dict(W=W_all, U=U_all, E=E_all, T=T_all,
                          S_start=S_start)
    return o, S


def la_chunk_forward(q, k, v, beta, g=None, gate="none", S0=None, C=64,
                     scale=1.0):
    """Chunkwise forms of linear attention read through a (preconditioned)
    query, App. D "Chunkwise parallel forms for preconditioned linear
    attention and its decayed variants".  q is the query the read-out uses
    (for the apply-to-query modes, the preconditioned query); per chunk:

      PLA (no decay):
          O = Q S^T + ((Q K^T) * M) V,       S <- S + V^T K
      P-Mamba-2 (scalar decay), gamma_r = prod_{j<=r in chunk} alpha_j:
          O = (gamma Q) S^T + ((Q K^T) * Gamma) V,
          Gamma_rj = gamma_r / gamma_j for r >= j, else 0,
          S <- gamma_C S + V^T ((gamma_C / gamma) K)
      PGLA (per-channel decay), Lam_r = prod_{j<=r in chunk} alpha_j,
      Gam_r = Lam_C / Lam_r, gam = Lam_C (all elementwise over d_k):
          O = (Q * Lam) S^T + (((Q * Lam)(K / Lam)^T) * M) V,
          S <- S Diag(gam) + V^T (K * Gam)

    M is the causal mask with the diagonal.  The paper prints these forms
    without a gain; the gain beta of S_t = alpha_t S_{t-1} + beta_t v_t k_t^T
    enters as V -> Diag(beta) V.  Returns (o (N,T,dv), S_T (N,dv,dk))."""
    q, k, v, beta = map(_f64, (q, k, v, beta))
    N, T, dk = k.shape
    dv = v.shape[2]
    S = np.zeros((N, dv, dk)) if S0 is None else _f64(S0).copy()
    o = np.empty((N, T, dv))
    for s, e in chunk_bounds(T, C):
        n = e - s
        Q, K = q[:, s:e], k[:, s:e]
        V = beta[:, s:e, None] * v[:, s:e]
        causal = np.tril(np.ones((n, n), bool))[None]
        St = np.swapaxes(S, 1, 2)                            # S^T (dk, dv)
        if gate == "none":
            o[:, s:e] = Q @ St + np.where(causal, Q @ np.swapaxes(K, 1, 2),
                                          0.0) @ V
            S = S + np.swapaxes(V, 1, 2) @ K
        elif gate == "scalar":
            gam = np.cumprod(np.exp(_f64(g)[:, s:e]), axis=1)     # (N, n)
            Gam = np.where(causal, gam[:, :, None] / gam[:, None, :], 0.0)
            o[:, s:e] = (gam[:, :, None] * Q) @ St + (
                (Q @ np.swapaxes(K, 1, 2)) * Gam) @ V
            gC = gam[:, -1]
            S = gC[:, None, None] * S + np.swapaxes(V, 1, 2) @ (
                (gC[:, None] / gam)[:, :, None] * K)
        elif gate == "channel":
            Lam = np.cumprod(np.exp(_f64(g)[:, s:e]), axis=1)     # (N, n, dk)
            QL = Q * Lam
            o[:, s:e] = QL @ St + np.where(
                causal, QL @ np.swapaxes(K / Lam, 1, 2), 0.0) @ V
            LC = Lam[:, -1:, :]
            S = S * LC + np.swapaxes(V, 1, 2) @ (K * (LC / Lam))
        else:
            raise ValueError(gate)
    return scale * o, S
