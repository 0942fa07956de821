"""The training pair on the GPU: pdn_chunk_fwd_train computes what
pdn_chunk_fwd computes, and pdn_chunk_bwd_train (reading the intermediates
the training forward left in the workspace) what pdn_chunk_bwd computes with
its own recompute.  Both pairs run the same kernels on the same values, so
the results must agree bit for bit; the backward paths are pinned to the
oracle in test_gpu_bwd.py."""
import numpy as np
import pytest

import pdn_inputs as pi

from gpu_util import to_device

pytestmark = pytest.mark.gpu

CASES = [
    # (io, gate, precond, dk, dv, T)
    ("bf16", "scalar", "squash", 128, 128, 200),
    ("bf16", "none", "squash", 128, 64, 64),
    ("bf16", "scalar", "identity", 64, 128, 130),
    ("bf16", "none", "external", 64, 64, 65),
    ("f32", "scalar", "squash", 64, 64, 200),
    ("bf16", "scalar", "squash", 128, 128, 1),
    ("bf16", "channel", "squash", 128, 128, 200),
    ("f32", "channel", "identity", 64, 64, 130),
]


def _run(spec, inp, precond, chunk=64):
    import torch
    import paper_2604_21100_amd as pdn
    d = to_device(inp, spec.io)
    sq = precond == "squash"
    kw = dict(g=d["g"], gate=spec.gate, precond=precond,
              beta_p=d["beta_p"] if sq else None, g_p=d["g_p"] if sq else None,
              log_a_scale=d["log_a_scale"] if sq else None,
              A0=d["A0"] if sq else None, S0=d["S0"],
              ktilde=d.get("ktilde") if precond == "external" else None,
              x=spec.x, scale=spec.scale, chunk=chunk)
    B, T, H = spec.B, spec.T, spec.H
    prob = pdn.make_problem(B, T, H, spec.dk, spec.dv, io=spec.io,
                            gate=spec.gate, precond=precond, x=spec.x,
                            scale=spec.scale, chunk=chunk)
    ws = torch.zeros(max(pdn.pdn_workspace_size(prob, True), 1),
                     dtype=torch.uint8, device="cuda")
    dST = torch.from_numpy((0.1 * np.random.default_rng(3).standard_normal(
        (B, H, spec.dk, spec.dv))).astype(np.float32)).cuda()
    ref_f = pdn.pdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], **kw)
    ref_b = pdn.pdn_chunk_bwd(d["q"], d["k"], d["v"], d["beta"], d["dO"],
                              dS_T=dST, **kw)
    got_f = pdn.pdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], workspace=ws,
                              train=True, **kw)
    got_b = pdn.pdn_chunk_bwd(d["q"], d["k"], d["v"], d["beta"], d["dO"],
                              dS_T=dST, workspace=ws, saved=True, **kw)
    again = pdn.pdn_chunk_bwd(d["q"], d["k"], d["v"], d["beta"], d["dO"],
                              dS_T=dST, workspace=ws, saved=True, **kw)
    torch.cuda.synchronize()
    return ref_f, ref_b, got_f, got_b, again


@pytest.mark.parametrize("chunk", [64, 32])
@pytest.mark.parametrize("io,gate,precond,dk,dv,T", CASES)
def test_training_pair_matches(io, gate, precond, dk, dv, T, chunk):
    import torch
    spec = pi.small_spec(io=io, gate=gate, dk=dk, dv=dv, T=T, s0="normal",
                         a0="lognormal" if precond == "squash" else "zero",
                         with_do=True)
    inp = pi.generate(spec, 77 + T)
    if precond == "external":
        rng = np.random.default_rng(5)
        kt = inp["k"] * rng.uniform(1 / 1.5, 1.5, inp["k"].shape)
        inp["ktilde"] = pi.round_bf16(kt) if io == "bf16" else kt.astype(np.float32)
    ref_f, ref_b, got_f, got_b, again = _run(spec, inp, precond, chunk)
    print(f"{io}/{gate}/{precond}/{dk}x{dv}/T={T}/chunk={chunk}")
    for a, b in zip(ref_f, got_f):
        if a is None:
            assert b is None
            continue
        assert torch.equal(a, b)
    assert set(ref_b) == set(got_b)
    for name in ref_b:
        assert torch.equal(ref_b[name], got_b[name]), name
        assert torch.equal(got_b[name], again[name]), name


def test_training_pair_bench_workload_sampled_heads():
    """The exact step bench.py times: the 1B PGDN layer (B=4, T=4096, H=16,
    d=128, bf16, scalar gate, squash, x=1.5) with the bench's seed and its
    dO ~ N(0, 1), through pdn_chunk_fwd_train + pdn_chunk_bwd_train.  At
    B*H = 64 the scans map 8 XCD groups x 4 value slabs; heads (0,0), (1,7)
    and (3,15) sit in different groups and batches.  Forward outputs, final
    states and every gradient of those heads are compared with the oracle's
    token recurrence and adjoint at the bf16 bar."""
    import dataclasses
    import torch
    import paper_2604_21100_amd as pdn
    from oracle import abi as oabi
    from gpu_util import rel_err, tol

    name = "pgdn_bf16_b4_t4096_h16_d128"
    spec = dataclasses.replace(pi.WORKLOADS[name], with_do=True)
    inp = pi.generate(spec, pi.WORKLOAD_SEEDS[name])
    d = to_device(inp, spec.io)
    kw = dict(g=d["g"], gate=spec.gate, beta_p=d["beta_p"], g_p=d["g_p"],
              log_a_scale=d["log_a_scale"], A0=d["A0"], S0=d["S0"], x=spec.x,
              scale=spec.scale)
    B, T, H = spec.B, spec.T, spec.H
    prob = pdn.make_problem(B, T, H, spec.dk, spec.dv, io=spec.io,
                            gate=spec.gate, x=spec.x, scale=spec.scale)
    ws = torch.empty(pdn.pdn_workspace_size(prob, True), dtype=torch.uint8,
                     device="cuda")
    o, S_T, A_T = pdn.pdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"],
                                    workspace=ws, train=True, **kw)
    grads = pdn.pdn_chunk_bwd(d["q"], d["k"], d["v"], d["beta"], d["dO"],
                              workspace=ws, saved=True, **kw)
    torch.cuda.synchronize()
    heads = [(0, 0), (1, 7), (3, 15)]
    cv = lambda t: t.float().cpu().numpy().astype(np.float64)  # noqa: E731
    rf = oabi.forward(inp, gate=spec.gate, x=spec.x, scale=spec.scale,
                      heads=heads)
    rb = oabi.backward(inp, gate=spec.gate, x=spec.x, scale=spec.scale,
                       heads=heads)
    o, S_T, A_T = cv(o), cv(S_T), cv(A_T)
    errs = {
        "o": rel_err(np.stack([o[b, :, h] for b, h in heads]), rf["o"]),
        "S_T": rel_err(np.stack([S_T[b, h] for b, h in heads]), rf["S_T"]),
        "A_T": rel_err(np.stack([A_T[b, h] for b, h in heads]), rf["A_T"]),
    }
    for key in ("dq", "dk", "dv", "dbeta", "dg", "dS0", "dbeta_p", "dg_p",
                "dA0"):
        g = cv(grads[key])
        gs = (np.stack([g[b, h] for b, h in heads]) if key in ("dS0", "dA0")
              else np.stack([g[b, :, h] for b, h in heads]))
        errs[key] = rel_err(gs, rb[key])
    msg = name + " train pair, heads (0,0) (1,7) (3,15): " + " ".join(
        f"{k}={v:.2e}" for k, v in errs.items())
    print(msg)
    assert errs["A_T"] < 1e-4, msg
    assert max(errs.values()) <= tol(spec.io), msg
