"""Reverse-mode derivative of the token recurrence, float64.  TEST
INFRASTRUCTURE ONLY (see the package header).

The paper gives the backward pass only as a sequence of kernels (App. C,
backward pseudocode); what it must compute is the exact gradient of the
forward recurrence of Eq. precond_end2end (with the gated forms of Sec. 3.5).
This module differentiates that recurrence by hand, one token at a time, in
reverse, with the forward states recomputed from checkpoints every
`ckpt` tokens.  It is pinned by central finite differences in the tests.

Per token t (paper orientation, S is (dv, dk)):
    A_t   = aP_t A_{t-1} + bP_t k_t^2            aP_t = exp(gP_t)
    r     = log A_t - mu,  s = r/(1+|r|),  B = exp(-log(x) s),  kt = B k_t
    Sbar  = alpha_t S_{t-1}  (S Diag(alpha_t) for the per-channel gate)
    p     = Sbar k_t,  e = beta_t (v_t - p),  S_t = Sbar + e kt^T
    o_t   = scale S_t q_t
"""
from __future__ import annotations

import numpy as np

from .recurrent import _f64, decay_state, preconditioner_scan, squash


def pdn_backward(q, k, v, beta, do, *, g=None, gate="none",
                 precond="squash", beta_p=None, g_p=None, mu=None, x=1.5,
                 kt_ext=None, S0=None, A0=None, scale=1.0, dS_T=None,
                 ckpt=64):
    """Gradients of sum_t <do_t, o_t> + <dS_T, S_T> with respect to every
    input.  Shapes as in `recurrent` (per-head layout).  Returns a dict with
    dq, dk, dv (N,T,d); dbeta, dg (N,T) or dg (N,T,dk); dS0 (N,dv,dk);
    and for precond="squash": dbeta_p, dg_p (N,T), dmu (N,), dA0 (N,dk),
    and dmu_abs (N,), the sum of the absolute values of dmu's terms;
    for precond="external": dkt (N,T,dk)."""
    q, k, v, beta, do = map(_f64, (q, k, v, beta, do))
    g = _f64(g)
    N, T, dk = k.shape
    dv_ = v.shape[2]
    if precond == "squash":
        mu = np.ones(N) if mu is None else _f64(mu)
        kt, A_all, _ = preconditioner_scan(k, beta_p, g_p, mu, x, A0)
        beta_p = _f64(beta_p)
        A_init = np.zeros((N, dk)) if A0 is None else _f64(A0)
    elif precond == "identity":
        kt = k
    else:
        kt = _f64(kt_ext)

    def alpha_at(t):
        return None if gate == "none" else np.exp(g[:, t])

    def step(S, t):
        a = alpha_at(t)
        Sbar = decay_state(S, a, gate)
        p = np.einsum("nvk,nk->nv", Sbar, k[:, t])
        e = beta[:, t, None] * (v[:, t] - p)
        return Sbar, p, e, Sbar + e[:, :, None] * kt[:, t, None, :]

    # forward pass, keeping the state before every ckpt-th token
    S = np.zeros((N, dv_, dk)) if S0 is None else _f64(S0).copy()
    ckpts = {}
    for t in range(T):
        if t % ckpt == 0:
            ckpts[t] = S.copy()
        S = step(S, t)[3]

    dq = np.zeros_like(q)
    dkk = np.zeros_like(k)
    dkt_all = np.zeros_like(k)
    dvv = np.zeros_like(v)
    dbeta = np.zeros((N, T))
    dg = None if gate == "none" else np.zeros_like(g)
    dS = np.zeros((N, dv_, dk)) if dS_T is None else _f64(dS_T).copy()

    for c0 in sorted(ckpts, reverse=True):
        c1 = min(c0 + ckpt, T)
        states = [ckpts[c0]]                      # S_{t-1} for t in [c0, c1)
        for t in range(c0, c1 - 1):
            states.append(step(states[-1], t)[3])
        for t in range(c1 - 1, c0 - 1, -1):
            S_prev = states[t - c0]
            Sbar, p, e, S_t = step(S_prev, t)
            # o_t = scale S_t q_t
            dS += scale * do[:, t, :, None] * q[:, t, None, :]
            dq[:, t] = scale * np.einsum("nvk,nv->nk", S_t, do[:, t])
            # S_t = Sbar + e kt^T
            de = np.einsum("nvk,nk->nv", dS, kt[:, t])
            dkt_all[:, t] = np.einsum("nvk,nv->nk", dS, e)
            # e = beta (v - p)
            dbeta[:, t] = np.einsum("nv,nv->n", de, v[:, t] - p)
            dvv[:, t] = beta[:, t, None] * de
            dp = -beta[:, t, None] * de
            # p = Sbar k
            dSbar = dS + dp[:, :, None] * k[:, t, None, :]
            dkk[:, t] += np.einsum("nvk,nv->nk", Sbar, dp)
            # Sbar = alpha S_prev ;  d/dg = alpha d/dalpha
            if gate == "scalar":
                dg[:, t] = np.einsum("nvk,nvk->n", dSbar, Sbar)
            elif gate == "channel":
                dg[:, t] = np.einsum("nvk,nvk->nk", dSbar, Sbar)
            dS = decay_state(dSbar, alpha_at(t), gate)

    out = dict(dq=dq, dv=dvv, dbeta=dbeta, dS0=dS)
    if gate != "none":
        out["dg"] = dg

    if precond == "identity":
        dkk += dkt_all
    elif precond == "external":
        out["dkt"] = dkt_all
    else:
        # kt = B(A_t) k_t and the A recurrence, in reverse
        lnx = np.log(x)
        dA = np.zeros((N, dk))
        dmu = np.zeros(N)
        dmu_abs = np.zeros(N)   # sum of |terms| of dmu: the scale of its rounding error
        dbeta_p = np.zeros((N, T))
        dg_p = np.zeros((N, T))
        m = mu.reshape(N, 1)
        for t in range(T - 1, -1, -1):
            A_t = A_all[:, t]
            A_prev = A_all[:, t - 1] if t > 0 else A_init
            Bt = squash(A_t, m, x)
            dkk[:, t] += Bt * dkt_all[:, t]
            dB = dkt_all[:, t] * k[:, t]
            ds = -lnx * Bt * dB
            pos = A_t > 0
            with np.errstate(divide="ignore", invalid="ignore"):
                r = np.log(A_t) - m
                dr = np.where(pos, ds / (1.0 + np.abs(r)) ** 2, 0.0)
                dA_tot = dA + np.where(pos, dr / A_t, 0.0)
            dmu -= dr.sum(axis=1)
            dmu_abs += np.abs(dr).sum(axis=1)
            dbeta_p[:, t] = np.einsum("nk,nk->n", dA_tot, k[:, t] ** 2)
            dkk[:, t] += 2.0 * beta_p[:, t, None] * k[:, t] * dA_tot
            a_p = np.ones(N) if g_p is None else np.exp(_f64(g_p)[:, t])
            dg_p[:, t] = a_p * np.einsum("nk,nk->n", dA_tot, A_prev)
            dA = a_p[:, None] * dA_tot
        out.update(dbeta_p=dbeta_p, dg_p=dg_p, dmu=dmu, dmu_abs=dmu_abs, dA0=dA)
    out["dk"] = dkk
    return out
