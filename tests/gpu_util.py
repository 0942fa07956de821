"""Helpers shared by the GPU tests: move seeded inputs to the device, run the
library through its C ABI, compare with the oracle."""
import numpy as np

IO_KEYS = ("q", "k", "v", "dO", "ktilde")


def to_device(inp, io):
    import torch
    out = {}
    for key, a in inp.items():
        if a is None:
            out[key] = None
            continue
        t = torch.from_numpy(np.ascontiguousarray(a))
        if key in IO_KEYS:
            t = t.to(torch.bfloat16 if io == "bf16" else torch.float32)
        out[key] = t.cuda()
    return out


def run_fwd(spec, inp, precond="squash", dev=None, **kw):
    """Forward on the GPU; returns float64 numpy (o, S_T, A_T)."""
    import torch
    import paper_2604_21100_amd as pdn
    d = dev if dev is not None else to_device(inp, spec.io)
    sq = precond == "squash"
    gram = precond in ("squash", "diag_sm", "atq")
    o, S_T, A_T = pdn.pdn_chunk_fwd(
        d["q"], d["k"], d["v"], d["beta"], g=d["g"], gate=spec.gate,
        precond=precond, beta_p=d["beta_p"] if gram else None,
        g_p=d["g_p"] if gram else None,
        log_a_scale=d["log_a_scale"] if sq else None,
        A0=d["A0"] if gram else None, S0=d["S0"],
        ktilde=d.get("ktilde") if precond == "external" else None,
        x=spec.x, scale=spec.scale, **kw)
    torch.cuda.synchronize()
    cv = (lambda t: None if t is None else t.float().cpu().numpy().astype(np.float64))
    return cv(o), cv(S_T), cv(A_T)


def rel_err(x, r):
    """max |x - r| / max |r| (normwise max error)."""
    x = np.asarray(x, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    den = np.abs(r).max()
    if den == 0:
        return float(np.abs(x).max())
    return float(np.abs(x - r).max() / den)


def tol(io):
    return 2e-2 if io == "bf16" else 1e-4
