"""C-ABI layout adapters and a per-head process pool for the oracle.  TEST
INFRASTRUCTURE ONLY (see the package header).

The C ABI stores per-token tensors as [B, T, H, d], scalars per token-head
as [B, T, H], the state as [B, H, dk, dv] (the transpose of the paper's S)
and the preconditioner state as [B, H, dk].  The oracle works per head
(N = B*H heads, paper orientation); these helpers convert, optionally for a
subset of heads only, so that full-size GPU runs can be checked on sampled
heads.
"""
from __future__ import annotations

import os
from concurrent.futures import ProcessPoolExecutor

import numpy as np

from . import adjoint, chunkwise, recurrent


def _sel(x, heads, tok):
    """Pick heads [(b, h), ...] from a [B, T, H, ...] (tok=True) or
    [B, H, ...] (tok=False) array -> [n, ...] float64."""
    if x is None:
        return None
    x = np.asarray(x)
    if tok:
        return np.stack([x[b, :, h] for b, h in heads]).astype(np.float64)
    return np.stack([x[b, h] for b, h in heads]).astype(np.float64)


def all_heads(B, H):
    return [(b, h) for b in range(B) for h in range(H)]


def head_inputs(inp, heads, gate, precond):
    """Per-head float64 views of an input dict produced by pdn_inputs."""
    d = dict(
        q=_sel(inp["q"], heads, True), k=_sel(inp["k"], heads, True),
        v=_sel(inp["v"], heads, True), beta=_sel(inp["beta"], heads, True),
        g=_sel(inp.get("g"), heads, True) if gate != "none" else None,
        beta_p=_sel(inp.get("beta_p"), heads, True),
        g_p=_sel(inp.get("g_p"), heads, True),
        mu=np.exp(np.array([float(inp["log_a_scale"][h]) for _, h in heads])),
        A0=_sel(inp.get("A0"), heads, False),
        S0=None,
        kt_ext=_sel(inp.get("ktilde"), heads, True)
        if precond == "external" else None,
        do=_sel(inp.get("dO"), heads, True),
    )
    S0 = inp.get("S0")
    if S0 is not None:
        d["S0"] = np.swapaxes(_sel(S0, heads, False), 1, 2)   # -> (dv, dk)
    return d


def forward(inp, *, gate, precond="squash", x=1.5, scale=1.0, heads=None,
            B=None, H=None, ridge=1.0, knorm="none"):
    """Token-recurrence forward for the selected heads.  Returns dict with
    o (n, T, dv), S_T (n, dk, dv) in ABI orientation, A_T (n, dk), kt."""
    if heads is None:
        heads = all_heads(B, H)
    d = head_inputs(inp, heads, gate, precond)
    r = recurrent.pdn_forward(
        d["q"], d["k"], d["v"], d["beta"], g=d["g"], gate=gate,
        precond=precond, beta_p=d["beta_p"], g_p=d["g_p"], mu=d["mu"], x=x,
        kt_ext=d["kt_ext"], S0=d["S0"], A0=d["A0"], scale=scale, ridge=ridge,
        knorm=knorm)
    r["S_T"] = np.swapaxes(r["S_T"], 1, 2)
    return r


def chunk_intermediates(inp, *, gate, precond="squash", x=1.5, scale=1.0,
                        C=64, heads=None, B=None, H=None):
    """Chunkwise-form intermediates (write key, T, W, U, E, chunk-start
    states in ABI orientation, preconditioner boundary states)."""
    if heads is None:
        heads = all_heads(B, H)
    d = head_inputs(inp, heads, gate, precond)
    A_bound = None
    if precond == "squash":
        kt, A_bound = chunkwise.preconditioner_chunkwise(
            d["k"], d["beta_p"], d["g_p"], d["mu"], x, C, d["A0"])
    elif precond == "identity":
        kt = d["k"]
    else:
        kt = d["kt_ext"]
    o, S_T, inter = chunkwise.chunk_forward(
        d["q"], d["k"], kt, d["v"], d["beta"], d["g"], gate, d["S0"], C,
        scale, keep=True)
    inter.update(o=o, S_T=np.swapaxes(S_T, 1, 2), kt=kt, A_bound=A_bound,
                 S_start=np.swapaxes(inter["S_start"], 2, 3))
    return inter


def backward(inp, *, gate, precond="squash", x=1.5, scale=1.0, heads=None,
             B=None, H=None, dS_T=None):
    """Adjoint for the selected heads; dS0 in ABI orientation, dmu turned
    into d logAScale per head (dlog_a_scale_h = mu_h * dmu_h)."""
    if heads is None:
        heads = all_heads(B, H)
    d = head_inputs(inp, heads, gate, precond)
    dST = None if dS_T is None else np.swapaxes(_sel(dS_T, heads, False), 1, 2)
    r = adjoint.pdn_backward(
        d["q"], d["k"], d["v"], d["beta"], d["do"], g=d["g"], gate=gate,
        precond=precond, beta_p=d["beta_p"], g_p=d["g_p"], mu=d["mu"], x=x,
        kt_ext=d["kt_ext"], S0=d["S0"], A0=d["A0"], scale=scale, dS_T=dST)
    r["dS0"] = np.swapaxes(r["dS0"], 1, 2)
    if "dmu" in r:
        r["dlog_a_scale"] = d["mu"] * r["dmu"]
        r["dlog_a_scale_abs"] = d["mu"] * r["dmu_abs"]
    return r


def _fwd_job(args):
    inp, kw, heads = args
    os.environ.setdefault("OMP_NUM_THREADS", "1")
    return forward(inp, heads=heads, **kw)


def pooled_forward(inp, heads, workers, **kw):
    """Run `forward` over head groups in a process pool (one head group per
    worker); returns the list of per-group results."""
    groups = [heads[i::workers] for i in range(workers)]
    groups = [g for g in groups if g]
    # ship only the selected heads' data to the workers
    with ProcessPoolExecutor(max_workers=len(groups)) as ex:
        return list(ex.map(_fwd_job, [(inp, kw, g) for g in groups]))
