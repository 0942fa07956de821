"""Token-by-token recurrences in float64.  TEST INFRASTRUCTURE ONLY (see the
package header): nothing in the product path imports this module.

Per-head layout used throughout the oracle (N = number of heads):
    q, k, kt   (N, T, dk)     v, o  (N, T, dv)
    beta, beta_p, g_p, scalar g     (N, T)
    per-channel g                   (N, T, dk)
    mu                              (N,)        mu = exp(logAScale) of the head
    S                               (N, dv, dk) the paper's orientation
    A                               (N, dk)     diagonal preconditioner state
"""
from __future__ import annotations

import numpy as np

F64 = np.float64


def _f64(x):
    return None if x is None else np.asarray(x, dtype=F64)


# --------------------------------------------------------------------------
# Stable diagonal preconditioner on the write key (Sec. 3.5, Eq.
# precond_end2end; decay/gain form App. E "ATQ vs ATK", App. D "ATK
# (stable) preconditioner recurrence").
# --------------------------------------------------------------------------
def squash(A, mu, x):
    """B = exp(-log(x) * s) with s = r / (1 + |r|) and r = log(A) - mu,
    elementwise (Eq. precond_end2end).  B lies in [1/x, x] and decreases
    as A grows.

    A channel whose keys have all been zero so far has A = 0 and
    r = -inf; the paper does not treat it, and we take the limit
    s -> -1, i.e. B = x (the largest gain)."""
    A = _f64(A)
    mu = _f64(mu)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.log(A) - mu
        s = np.where(A > 0.0, r / (1.0 + np.abs(r)), -1.0)
    return np.exp(-np.log(F64(x)) * s)


def preconditioner_scan(k, beta_p, g_p, mu, x, A0=None):
    """Diagonal key-Gram recurrence and preconditioned write key.

        A_t  = alpha^P_t A_{t-1} + beta^P_t (k_t * k_t),  alpha^P_t = exp(g^P_t)
        kt_t = B(A_t) * k_t

    (Eq. precond_end2end; the current A_t, not A_{t-1}, and no
    Sherman-Morrison normalisation: App. E "Stable parameterization").
    g_p = None means alpha^P = 1 (Eq. diag_gram's undecayed sum).

    Returns (kt (N,T,dk), A_all (N,T,dk) with A_all[:, t] = A_t, A_T (N,dk)).
    """
    k = _f64(k)
    N, T, dk = k.shape
    beta_p = _f64(beta_p)
    A = np.zeros((N, dk)) if A0 is None else _f64(A0).copy()
    mu = _f64(mu).reshape(N, 1)
    kt = np.empty_like(k)
    A_all = np.empty_like(k)
    for t in range(T):
        a_p = 1.0 if g_p is None else np.exp(_f64(g_p)[:, t])[:, None]
        A = a_p * A + beta_p[:, t, None] * (k[:, t] * k[:, t])
        A_all[:, t] = A
        kt[:, t] = squash(A, mu, x) * k[:, t]
    return kt, A_all, A


def gram_states(k, beta_p, g_p, A0=None):
    """The diagonal key-Gram recurrence alone (Eq. diag_gram with the decay
    and gain of Eq. precond_end2end):

        A_t = alpha^P_t A_{t-1} + beta^P_t (k_t * k_t)

    Returns (A_prev (N,T,dk) with A_prev[:, t] = A_{t-1}, A_all (N,T,dk)
    with A_all[:, t] = A_t, A_T (N,dk))."""
    k = _f64(k)
    N, T, dk = k.shape
    beta_p = _f64(beta_p)
    A = np.zeros((N, dk)) if A0 is None else _f64(A0).copy()
    A_prev = np.empty_like(k)
    A_all = np.empty_like(k)
    for t in range(T):
        A_prev[:, t] = A
        a_p = 1.0 if g_p is None else np.exp(_f64(g_p)[:, t])[:, None]
        A = a_p * A + beta_p[:, t, None] * (k[:, t] * k[:, t])
        A_all[:, t] = A
    return A_prev, A_all, A


def sm_write_key(k, A_prev, lam):
    """Write key of the diagonal Sherman-Morrison ("unstable ATK") form, App.
    D "ATK (unstable) preconditioner recurrence":

        kt_t = P_t k_t / (1 + k_t^T P_t k_t),  P_t = Diag(A_{t-1} + lam)^{-1}
    """
    k, A_prev = _f64(k), _f64(A_prev)
    pk = k / (A_prev + lam)
    return pk / (1.0 + np.sum(k * pk, axis=-1, keepdims=True))


# --------------------------------------------------------------------------
# Main recurrence with distinct read key k and write key kt.
# --------------------------------------------------------------------------
def decay_state(S, alpha, gate):
    """alpha_t S_{t-1}: a scalar for the Gated-DeltaNet form; for the KDA
    form alpha_t is a d_k-vector acting on the key side, S Diag(alpha)
    (App. D "Diagonally-decayed PDN")."""
    if gate == "none":
        return S
    if gate == "scalar":
        return alpha[:, None, None] * S
    if gate == "channel":
        return S * alpha[:, None, :]
    raise ValueError(gate)


def delta_rule(q, k, kt, v, beta, g=None, gate="none", S0=None, scale=1.0,
               return_states=False):
    """Preconditioned (gated) delta rule, one token at a time:

        S_t = alpha_t S_{t-1} + beta_t (v_t - alpha_t S_{t-1} k_t) kt_t^T
        o_t = scale * S_t q_t

    (Eq. precond_end2end for alpha = 1; PGDN/PKDA by replacing S_{t-1} with
    alpha_t S_{t-1}, Sec. 3.5 and App. E Lemma "Eigenvalues of the GDN/PGDN
    transition").  k is the read key, kt the write key.

    Returns (o (N,T,dv), S_T (N,dv,dk)[, S_all (N,T,dv,dk)])."""
    q, k, kt, v, beta = map(_f64, (q, k, kt, v, beta))
    g = _f64(g)
    N, T, dk = k.shape
    dv = v.shape[2]
    S = np.zeros((N, dv, dk)) if S0 is None else _f64(S0).copy()
    o = np.empty((N, T, dv))
    S_all = np.empty((N, T, dv, dk)) if return_states else None
    for t in range(T):
        alpha = None if gate == "none" else np.exp(g[:, t])
        Sbar = decay_state(S, alpha, gate)
        pred = np.einsum("nvk,nk->nv", Sbar, k[:, t])          # read: S k
        err = beta[:, t, None] * (v[:, t] - pred)
        S = Sbar + err[:, :, None] * kt[:, t, None, :]          # write: e kt^T
        o[:, t] = scale * np.einsum("nvk,nk->nv", S, q[:, t])
        if return_states:
            S_all[:, t] = S
    if return_states:
        return o, S, S_all
    return o, S


def linear_attention(q, k, v, beta, g=None, gate="none", S0=None, scale=1.0):
    """(Gated) linear attention, one token at a time:

        S_t = alpha_t S_{t-1} + beta_t v_t k_t^T
        o_t = scale * S_t q_t

    (Sec. 2's linear attention; with a scalar alpha the Mamba-2 form, with
    a per-channel alpha acting as S Diag(alpha) the GLA form of App. E "ATQ
    vs ATK").  The apply-to-query modes pass the preconditioned query as q.

    Returns (o (N,T,dv), S_T (N,dv,dk))."""
    q, k, v, beta = map(_f64, (q, k, v, beta))
    g = _f64(g)
    N, T, dk = k.shape
    dv = v.shape[2]
    S = np.zeros((N, dv, dk)) if S0 is None else _f64(S0).copy()
    o = np.empty((N, T, dv))
    for t in range(T):
        alpha = None if gate == "none" else np.exp(g[:, t])
        S = decay_state(S, alpha, gate) + beta[:, t, None, None] * (
            v[:, t, :, None] * k[:, t, None, :])
        o[:, t] = scale * np.einsum("nvk,nk->nv", S, q[:, t])
    return o, S


def knorm_factor(k, kt, beta, g, gate, knorm):
    """Normalisation factor on the squash write key (App. E "Stable
    parameterization", ablation table), with m_t = k_t^T B_t k_t = k_t . kt_t:
        "none" 1,  "m" 1/m_t,  "1pm" 1/(1 + m_t),
        "beta" beta_t / (alpha_t + beta_t m_t)   (alpha_t = exp(g_t), scalar
               gate; 1 without a gate)
    Returns the (N, T, 1) factor."""
    m = np.sum(_f64(k) * _f64(kt), axis=-1, keepdims=True)
    if knorm == "none":
        return np.ones_like(m)
    if knorm == "m":
        return 1.0 / m
    if knorm == "1pm":
        return 1.0 / (1.0 + m)
    if knorm == "beta":
        if gate == "channel":
            raise ValueError("the beta factor needs a scalar decay")
        al = np.ones_like(m) if gate == "none" else np.exp(_f64(g))[..., None]
        b = _f64(beta)[..., None]
        return b / (al + b * m)
    raise ValueError(knorm)


def pdn_forward(q, k, v, beta, *, g=None, gate="none", precond="squash",
                beta_p=None, g_p=None, mu=None, x=1.5, kt_ext=None, S0=None,
                A0=None, scale=1.0, ridge=1.0, knorm="none"):
    """End-to-end token recurrence for PDN / PGDN / PKDA and the other
    preconditioner realisations.

    precond = "squash"    write key from Eq. precond_end2end
              "identity"  kt = k (plain DeltaNet / GDN / KDA)
              "external"  kt supplied by the caller (any write key)
              "diag_sm"   Sherman-Morrison write key from A_{t-1} + ridge
                          (sm_write_key), then the delta rule
              "atq"       linear attention read through the preconditioned
                          query q_t / (A_t + ridge) (App. D "ATQ
                          preconditioner recurrence"); kt = k
    knorm (squash only): the normalisation factor of knorm_factor.
    Returns dict(o, S_T, A_T, kt)."""
    k = _f64(k)
    N = k.shape[0]
    A_T = None
    if precond == "squash":
        if mu is None:
            mu = np.ones(N)
        kt, _, A_T = preconditioner_scan(k, beta_p, g_p, mu, x, A0)
        kt = kt * knorm_factor(k, kt, beta, g, gate, knorm)
    elif precond == "identity":
        kt = k
    elif precond == "external":
        kt = _f64(kt_ext)
    elif precond == "diag_sm":
        A_prev, _, A_T = gram_states(k, beta_p, g_p, A0)
        kt = sm_write_key(k, A_prev, ridge)
    elif precond == "atq":
        _, A_all, A_T = gram_states(k, beta_p, g_p, A0)
        qt = _f64(q) / (A_all + ridge)
        o, S_T = linear_attention(qt, k, v, beta, g, gate, S0, scale)
        return dict(o=o, S_T=S_T, A_T=A_T, kt=k)
    else:
        raise ValueError(precond)
    o, S_T = delta_rule(q, k, kt, v, beta, g, gate, S0, scale)
    return dict(o=o, S_T=S_T, A_T=A_T, kt=kt)


# --------------------------------------------------------------------------
# Oracle-only modes of Sec. 3.1 / 3.3 (pins, not GPU targets).  One head,
# S0 = 0, beta = 1, no gate unless stated.
# --------------------------------------------------------------------------
def exact_gram_pdn(k, v, q, lam):
    """PDN with the exact inverse key Gram (Eq. atk_update):

        P_0 = I / lam,  kt_t = P_{t-1} k_t / (1 + k_t^T P_{t-1} k_t)
        S_t = S_{t-1} + (v_t - S_{t-1} k_t) kt_t^T,  o_t = S_t q_t
        P_t = P_{t-1} - P_{t-1} k_t k_t^T P_{t-1} / (1 + k_t^T P_{t-1} k_t)

    (the Sherman-Morrison update of P_t = G_t^{-1}, App. B "MesaNet
    parallelization").  Inputs (T, d); returns (S_all (T,dv,dk),
    kt (T,dk), P_all (T,dk,dk), o (T,dv))."""
    k, v, q = map(_f64, (k, v, q))
    T, dk = k.shape
    dv = v.shape[1]
    P = np.eye(dk) / lam
    S = np.zeros((dv, dk))
    S_all = np.empty((T, dv, dk))
    P_all = np.empty((T, dk, dk))
    kts = np.empty((T, dk))
    o = np.empty((T, dv))
    for t in range(T):
        Pk = P @ k[t]
        denom = 1.0 + k[t] @ Pk
        kt = Pk / denom
        S = S + np.outer(v[t] - S @ k[t], kt)
        P = P - np.outer(Pk, Pk) / denom
        S_all[t], P_all[t], kts[t] = S, P, kt
        o[t] = S @ q[t]
    return S_all, kts, P_all, o


def diag_sm_pdn(k, v, q, lam, beta=None, beta_p=None, g_p=None, A0=None):
    """Diagonal-Gram PDN in Sherman-Morrison form (the 'unstable ATK' of
    App. D and App. E):

        kt_t = (A_{t-1}+lam)^{-1} k_t / (1 + k_t^T (A_{t-1}+lam)^{-1} k_t)
        A_t  = alpha^P_t A_{t-1} + beta^P_t k_t * k_t     (Eq. diag_gram)
        S_t  = S_{t-1} + beta_t (v_t - S_{t-1} k_t) kt_t^T

    Inputs (T, d); beta, beta_p default to 1, g_p to 0.  Returns
    (S_all (T,dv,dk), kt (T,dk), o (T,dv))."""
    k, v, q = map(_f64, (k, v, q))
    T, dk = k.shape
    dv = v.shape[1]
    beta = np.ones(T) if beta is None else _f64(beta)
    beta_p = np.ones(T) if beta_p is None else _f64(beta_p)
    A = np.zeros(dk) if A0 is None else _f64(A0).copy()
    S = np.zeros((dv, dk))
    S_all = np.empty((T, dv, dk))
    kts = np.empty((T, dk))
    o = np.empty((T, dv))
    for t in range(T):
        pk = k[t] / (A + lam)
        kt = pk / (1.0 + k[t] @ pk)
        a_p = 1.0 if g_p is None else np.exp(g_p[t])
        A = a_p * A + beta_p[t] * k[t] * k[t]
        S = S + beta[t] * np.outer(v[t] - S @ k[t], kt)
        S_all[t], kts[t] = S, kt
        o[t] = S @ q[t]
    return S_all, kts, o


def atq_pla(k, v, q, lam, beta=None, g=None):
    """Preconditioned linear attention, apply-to-query, diagonal Gram
    (Eq. atq_readout with G replaced by its diagonal, Eq. diag_gram;
    P-Mamba-2 when a scalar log-decay g is given, App. E "ATQ vs ATK"):

        C_t = alpha_t C_{t-1} + beta_t v_t k_t^T,  A_t = A_{t-1} + k_t * k_t
        o_t = C_t ((A_t + lam)^{-1} * q_t)

    Returns (M_all (T,dv,dk), o (T,dv)) where M_t = C_t Diag(A_t+lam)^{-1}
    is the effective read-out map."""
    k, v, q = map(_f64, (k, v, q))
    T, dk = k.shape
    dv = v.shape[1]
    beta = np.ones(T) if beta is None else _f64(beta)
    A = np.zeros(dk)
    C = np.zeros((dv, dk))
    M_all = np.empty((T, dv, dk))
    o = np.empty((T, dv))
    for t in range(T):
        a = 1.0 if g is None else np.exp(g[t])
        C = a * C + beta[t] * np.outer(v[t], k[t])
        A = A + k[t] * k[t]
        M_all[t] = C / (A + lam)[None, :]
        o[t] = C @ (q[t] / (A + lam))
    return M_all, o
