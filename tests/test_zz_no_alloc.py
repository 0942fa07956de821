"""The no-allocation forward (pdn_chunk_fwd_noalloc) on the GPU: through the
C ABI it must give what pdn_chunk_fwd gives with a caller workspace, on two
calls in a row of which the second is smaller (the shared per-device
scratch keeps the first call's contents), and on a third call of the first
size after it."""
import numpy as np
import pytest

import pdn_inputs as pi

from gpu_util import to_device

pytestmark = pytest.mark.gpu

CASES = [
    # first call, then a smaller one: (io, gate, precond, B, T, H, dk, dv)
    (("bf16", "scalar", "squash", 2, 700, 4, 128, 128),
     ("bf16", "scalar", "squash", 1, 130, 2, 128, 128)),
    (("bf16", "channel", "squash", 1, 1000, 3, 128, 128),
     ("bf16", "channel", "squash", 1, 65, 1, 128, 128)),
    (("f32", "none", "identity", 2, 300, 2, 64, 64),
     ("f32", "none", "identity", 1, 1, 1, 64, 64)),
]


def _case(io, gate, precond, B, T, H, dk, dv, seed):
    spec = pi.small_spec(io=io, gate=gate, B=B, T=T, H=H, dk=dk, dv=dv,
                         s0="normal",
                         a0="lognormal" if precond == "squash" else "zero")
    return spec, precond, to_device(pi.generate(spec, seed), io)


def _kw(spec, precond, d):
    sq = precond == "squash"
    return dict(g=d["g"], gate=spec.gate, precond=precond,
                beta_p=d["beta_p"] if sq else None,
                g_p=d["g_p"] if sq else None,
                log_a_scale=d["log_a_scale"] if sq else None,
                A0=d["A0"] if sq else None, S0=d["S0"], x=spec.x,
                scale=spec.scale)


def _both(spec, precond, d):
    import torch
    import paper_2604_21100_amd as pdn
    kw = _kw(spec, precond, d)
    ref = pdn.pdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], **kw)
    o = torch.full_like(ref[0], float("nan"))
    S_T = torch.full_like(ref[1], float("nan"))
    A_T = None if ref[2] is None else torch.full_like(ref[2], float("nan"))
    got = pdn.pdn_chunk_fwd_noalloc(d["q"], d["k"], d["v"], d["beta"], o=o,
                                    S_T=S_T, A_T=A_T, **kw)
    torch.cuda.synchronize()
    return ref, got


@pytest.mark.parametrize("first,second", CASES)
def test_noalloc_matches_forward(first, second):
    import torch
    big = _case(*first, seed=11)
    small = _case(*second, seed=12)
    for tag, (spec, precond, d) in (("first", big), ("second, smaller", small),
                                    ("third, first size again", big)):
        print(f"no-alloc {tag}: {spec.io}/{spec.gate}/{precond} "
              f"B={spec.B} T={spec.T} H={spec.H} dk={spec.dk} dv={spec.dv}",
              flush=True)
        ref, got = _both(spec, precond, d)
        for a, b in zip(ref, got):
            if a is None:
                assert b is None
                continue
            assert torch.equal(a, b), tag
