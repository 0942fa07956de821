"""GPU parity of the sequence-split state scan: with few heads the forward
scan runs in S >= 3 segments (segment 0 from S0, the middle segments' local
end states and d_k x d_k transitions from zero / the identity, the composed
exact starts, then segments 1 .. S - 1 again; see pdn_scan_segments in
pdn.h).  Every case here is a shape the library splits (asserted through
pdn_scan_segments) and is compared with the float64 oracle's token
recurrence, which knows nothing of segments: forward outputs and final
states on every head, the backward (whose forward recompute splits the same
way) on every gradient, and the training pair bit for bit against the
recompute path."""
import numpy as np
import pytest

import pdn_inputs as pi
from oracle import abi as oabi

from gpu_util import rel_err, run_fwd, tol

pytestmark = pytest.mark.gpu

CASES = [
    # (io, gate, precond, dk, dv, H, T): segments chosen by the library
    ("bf16", "scalar", "squash", 128, 128, 2, 1000),    # S = 4, ragged tail
    ("bf16", "channel", "squash", 128, 128, 2, 1000),
    ("bf16", "none", "identity", 64, 64, 2, 700),        # S = 3
    ("bf16", "scalar", "external", 64, 128, 3, 1000),
    ("bf16", "scalar", "squash", 128, 128, 1, 2112),     # S = 9, whole chunks
    ("f32", "scalar", "squash", 64, 64, 2, 700),
    ("f32", "channel", "identity", 64, 64, 1, 900),
]


def _spec_inputs(io, gate, precond, dk, dv, H, T, seed, with_do=False):
    spec = pi.small_spec(io=io, gate=gate, dk=dk, dv=dv, B=1, H=H, T=T,
                         s0="normal",
                         a0="lognormal" if precond == "squash" else "zero",
                         with_do=with_do)
    inp = pi.generate(spec, seed)
    if precond == "external":
        rng = np.random.default_rng(seed + 1)
        kt = inp["k"] * rng.uniform(1 / 1.5, 1.5, inp["k"].shape)
        inp["ktilde"] = pi.round_bf16(kt) if io == "bf16" else kt.astype(np.float32)
    return spec, inp


def _segments(spec, precond):
    import paper_2604_21100_amd as pdn
    return pdn.pdn_scan_segments(pdn.make_problem(
        spec.B, spec.T, spec.H, spec.dk, spec.dv, io=spec.io, gate=spec.gate,
        precond=precond))


@pytest.mark.parametrize("io,gate,precond,dk,dv,H,T", CASES)
def test_split_forward_all_heads(io, gate, precond, dk, dv, H, T):
    spec, inp = _spec_inputs(io, gate, precond, dk, dv, H, T, 900 + T)
    S = _segments(spec, precond)
    assert S >= 3
    o, S_T, A_T = run_fwd(spec, inp, precond)
    ref = oabi.forward(inp, gate=gate, precond=precond, x=spec.x,
                       scale=spec.scale, B=1, H=H)
    e_o = rel_err(np.stack([o[0, :, h] for h in range(H)]), ref["o"])
    e_s = rel_err(S_T.reshape(H, dk, dv), ref["S_T"])
    msg = f"split S={S} {io}/{gate}/{precond}/{dk}x{dv} H={H} T={T}: err(o)={e_o:.2e} err(S_T)={e_s:.2e}"
    print(msg)
    assert max(e_o, e_s) <= tol(io), msg
    if precond == "squash":
        assert rel_err(A_T.reshape(H, dk), ref["A_T"]) <= 1e-4


def test_split_forward_atq():
    """Linear attention with the preconditioned query (forward only): the
    transition of a segment is then a pure decay."""
    spec, inp = _spec_inputs("bf16", "scalar", "atq", 128, 128, 2, 1000, 77)
    assert _segments(spec, "atq") >= 3
    o, S_T, _ = run_fwd(spec, inp, "atq", ridge=1.0)
    ref = oabi.forward(inp, gate="scalar", precond="atq", x=spec.x,
                       scale=spec.scale, B=1, H=2, ridge=1.0)
    e_o = rel_err(np.stack([o[0, :, h] for h in range(2)]), ref["o"])
    e_s = rel_err(S_T.reshape(2, 128, 128), ref["S_T"])
    print(f"split atq err(o)={e_o:.2e} err(S_T)={e_s:.2e}")
    assert max(e_o, e_s) <= tol("bf16")


@pytest.mark.parametrize("io,gate,precond,dk,dv,H,T", CASES)
def test_split_backward_all_heads(io, gate, precond, dk, dv, H, T):
    from test_gpu_bwd import compare
    spec, inp = _spec_inputs(io, gate, precond, dk, dv, H, T, 950 + T, with_do=True)
    assert _segments(spec, precond) >= 3
    dS_T = (0.1 * np.random.default_rng(4).standard_normal(
        (1, H, dk, dv))).astype(np.float32)
    compare(spec, inp, precond, dS_T, tag=f"split bwd {io}/{gate}/{precond}/{dk}x{dv} H={H} T={T}")


@pytest.mark.parametrize("io,gate,precond,dk,dv,H,T", CASES[:5])
def test_split_training_pair_matches(io, gate, precond, dk, dv, H, T):
    import torch
    from test_gpu_train import _run
    spec, inp = _spec_inputs(io, gate, precond, dk, dv, H, T, 990 + T, with_do=True)
    assert _segments(spec, precond) >= 3
    ref_f, ref_b, got_f, got_b, again = _run(spec, inp, precond)
    for a, b in zip(ref_f, got_f):
        if a is None:
            assert b is None
            continue
        assert torch.equal(a, b)
    for name in ref_b:
        assert torch.equal(ref_b[name], got_b[name]), name
        assert torch.equal(got_b[name], again[name]), name
