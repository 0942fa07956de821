"""GPU parity of the backward pass (HIP kernels through the C ABI) against
the float64 oracle adjoint on the same seeded inputs.

Every gradient is compared with max|x - r| / max|r|: <= 1e-4 for fp32 io and
<= 2e-2 for bf16 io (the bar the forward outputs meet, applied to each
gradient).  The one exception is d logAScale, a sum over every token and
key channel of terms of both signs (the squash gain depends on mu through
r_t = log A_t - mu): its sum cancels to 0.1 - 0.7 % of the sum of its
terms' magnitudes, so its error is measured against that magnitude, the
scale of the standard bound for a rounded sum (error <= n u sum |x_i|)."""
import numpy as np
import pytest

import pdn_inputs as pi
from oracle import abi as oabi

from gpu_util import rel_err, to_device, tol

pytestmark = pytest.mark.gpu

NAMES = ["dq", "dk", "dv", "dbeta", "dg", "dS0", "dbeta_p", "dg_p",
         "dlog_a_scale", "dA0", "dktilde"]


def _heads(x, B, H):
    """[B, T, H, ...] -> [B*H, T, ...]"""
    x = np.asarray(x, dtype=np.float64)
    return np.stack([x[b, :, h] for b in range(B) for h in range(H)])


def run_bwd(spec, inp, precond="squash", dS_T=None, chunk=64):
    import torch
    import paper_2604_21100_amd as pdn
    d = to_device(inp, spec.io)
    sq = precond == "squash"
    dST = None if dS_T is None else torch.from_numpy(dS_T).cuda()
    out = pdn.pdn_chunk_bwd(
        d["q"], d["k"], d["v"], d["beta"], d["dO"], g=d["g"], gate=spec.gate,
        precond=precond, beta_p=d["beta_p"] if sq else None,
        g_p=d["g_p"] if sq else None,
        log_a_scale=d["log_a_scale"] if sq else None,
        A0=d["A0"] if sq else None, S0=d["S0"],
        ktilde=d.get("ktilde") if precond == "external" else None,
        dS_T=dST, x=spec.x, scale=spec.scale, chunk=chunk)
    torch.cuda.synchronize()
    return {k: v.float().cpu().numpy().astype(np.float64) for k, v in out.items()}


def compare(spec, inp, precond="squash", dS_T=None, heads=None, tag="", chunk=64):
    got = run_bwd(spec, inp, precond, dS_T, chunk)
    B, H = spec.B, spec.H
    if heads is None:
        heads = oabi.all_heads(B, H)
    ref = oabi.backward(inp, gate=spec.gate, precond=precond, x=spec.x,
                        scale=spec.scale, heads=heads, B=B, H=H, dS_T=dS_T)
    errs = {}
    for name in NAMES:
        if name not in got:
            continue
        g = got[name]
        if name == "dlog_a_scale":
            r = np.zeros(H)
            scale = np.zeros(H)
            for n, (b, h) in enumerate(heads):
                r[h] += ref["dlog_a_scale"][n]
                scale[h] += ref["dlog_a_scale_abs"][n]
            if len(heads) != B * H:
                continue
            errs[name] = float(np.abs(np.asarray(g, np.float64) - r).max() / scale.max())
            continue
        key = {"dktilde": "dkt"}.get(name, name)
        r = ref[key]
        if name in ("dS0", "dA0"):
            gs = np.stack([g[b, h] for b, h in heads])
        else:
            gs = np.stack([g[b, :, h] for b, h in heads])
        errs[name] = rel_err(gs, r)
    msg = f"{tag} " + " ".join(f"{k}={v:.2e}" for k, v in errs.items())
    print(msg)
    bad = {k: v for k, v in errs.items() if v > tol(spec.io)}
    assert not bad, msg
    return errs


SMALL = [
    # (io, gate, precond, dk, dv)
    ("bf16", "scalar", "squash", 128, 128),
    ("bf16", "none", "squash", 128, 128),
    ("bf16", "scalar", "identity", 128, 64),
    ("bf16", "none", "external", 64, 128),
    ("bf16", "scalar", "squash", 64, 64),
    ("f32", "scalar", "squash", 64, 64),
    ("f32", "none", "identity", 64, 64),
    ("f32", "scalar", "external", 64, 64),
    ("bf16", "channel", "squash", 128, 128),
    ("bf16", "channel", "identity", 128, 64),
    ("bf16", "channel", "external", 64, 128),
    ("bf16", "channel", "squash", 64, 64),
    ("f32", "channel", "squash", 64, 64),
    ("f32", "channel", "identity", 64, 64),
]


@pytest.mark.parametrize("io,gate,precond,dk,dv", SMALL)
def test_bwd_small_all_heads(io, gate, precond, dk, dv):
    """Several chunks plus a ragged tail (T = 200), every head, nonzero S0,
    A0 and dS_T."""
    spec = pi.small_spec(io=io, gate=gate, dk=dk, dv=dv, s0="normal",
                         a0="lognormal" if precond == "squash" else "zero",
                         with_do=True)
    inp = pi.generate(spec, 21)
    if precond == "external":
        rng = np.random.default_rng(6)
        kt = inp["k"] * rng.uniform(1 / 1.5, 1.5, inp["k"].shape)
        inp["ktilde"] = pi.round_bf16(kt) if io == "bf16" else kt.astype(np.float32)
    dS_T = (0.1 * np.random.default_rng(8).standard_normal(
        (spec.B, spec.H, dk, dv))).astype(np.float32)
    compare(spec, inp, precond, dS_T, tag=f"{io}/{gate}/{precond}/{dk}x{dv}")


@pytest.mark.parametrize("T", [1, 64, 65, 80, 114, 127, 130])
def test_bwd_sequence_lengths(T):
    """Last chunks of 1, 16 (a whole first segment of 16 tokens), 50 (into
    the fourth segment) and 63 tokens, and whole chunks."""
    spec = pi.small_spec(T=T, B=1, H=2, gate="scalar", dk=128, dv=128,
                         with_do=True)
    compare(spec, pi.generate(spec, 300 + T), tag=f"T={T}")


def test_bwd_zero_key_channels():
    """Key channels that are exactly zero with a zero initial state keep the
    preconditioner state at A = 0 there: the squash gain is x and has no
    derivative (the A <= 0 case of the gain), on both sides."""
    spec = pi.small_spec(gate="scalar", dk=128, dv=128, with_do=True, a0="zero")
    inp = pi.generate(spec, 41)
    inp["k"][..., ::7] = 0.0
    compare(spec, inp, tag="zero key channels")


def test_bwd_beta_range_and_squash_coverage():
    spec = pi.small_spec(gate="scalar", dk=128, dv=128, with_do=True,
                         beta_max=2.0, key_aniso=1.0, betap_logspan=2.0)
    compare(spec, pi.generate(spec, 31), tag="beta02/aniso")


@pytest.mark.parametrize("T", [1, 65, 114, 130])
def test_bwd_channel_gate_sequence_lengths(T):
    spec = pi.small_spec(T=T, B=1, H=2, gate="channel", dk=128, dv=128,
                         with_do=True)
    compare(spec, pi.generate(spec, 500 + T), tag=f"channel T={T}")


def test_bwd_strong_channel_gate():
    """Per-channel log-decays 15x the default (products of decay ratios
    across a chunk span many orders of magnitude), with anisotropic keys."""
    spec = pi.small_spec(gate="channel", dk=128, dv=128, with_do=True,
                         gate_strength=1.5, key_aniso=1.0)
    compare(spec, pi.generate(spec, 33), tag="strong channel gate")


def test_bwd_deterministic():
    spec = pi.small_spec(B=2, H=3, T=150, gate="scalar", with_do=True)
    inp = pi.generate(spec, 41)
    a = run_bwd(spec, inp)
    b = run_bwd(spec, inp)
    for key in a:
        assert np.array_equal(a[key], b[key]), key


def test_bwd_pkda_workload_sampled_heads():
    """The PKDA layer (B=2, T=8192, H=16, d=128, per-channel gate, N(0, 0.1)
    initial state) with an upstream dO ~ N(0, 1) drawn after the forward
    inputs: two heads recomputed by the oracle adjoint end to end."""
    import dataclasses
    name = "pkda_bf16_b2_t8192_h16_d128"
    spec = dataclasses.replace(pi.WORKLOADS[name], with_do=True)
    inp = pi.generate(spec, pi.WORKLOAD_SEEDS[name])
    compare(spec, inp, heads=[(0, 3), (1, 12)], tag=name + "+bwd")


def test_bwd_full_workload_sampled_heads():
    """The long-context PGDN workload (B=1, T=32768, H=16, d=128): two heads
    recomputed by the oracle adjoint end to end."""
    name = "pgdn_fwdbwd_bf16_b1_t32768_h16_d128"
    spec = pi.WORKLOADS[name]
    inp = pi.generate(spec, pi.WORKLOAD_SEEDS[name])
    compare(spec, inp, heads=[(0, 0), (0, 15)], tag=name)


CHUNK32 = [
    # (io, gate, precond, dk, dv): the backward with 32-token chunks
    ("bf16", "scalar", "squash", 128, 128),
    ("bf16", "none", "squash", 128, 64),
    ("bf16", "channel", "squash", 128, 128),
    ("bf16", "scalar", "identity", 64, 128),
    ("bf16", "channel", "external", 128, 64),
    ("f32", "scalar", "squash", 64, 64),
    ("f32", "channel", "identity", 64, 64),
    ("f32", "none", "external", 64, 64),
]


@pytest.mark.parametrize("io,gate,precond,dk,dv", CHUNK32)
def test_bwd_chunk32_all_heads(io, gate, precond, dk, dv):
    """chunk = 32: T = 200 (six chunks and a ragged tail of 8), every head,
    nonzero S0, A0 and dS_T, every gradient against the oracle adjoint."""
    spec = pi.small_spec(io=io, gate=gate, dk=dk, dv=dv, s0="normal",
                         a0="lognormal" if precond == "squash" else "zero",
                         with_do=True)
    inp = pi.generate(spec, 23)
    if precond == "external":
        rng = np.random.default_rng(6)
        kt = inp["k"] * rng.uniform(1 / 1.5, 1.5, inp["k"].shape)
        inp["ktilde"] = pi.round_bf16(kt) if io == "bf16" else kt.astype(np.float32)
    dS_T = (0.1 * np.random.default_rng(8).standard_normal(
        (spec.B, spec.H, dk, dv))).astype(np.float32)
    compare(spec, inp, precond, dS_T, tag=f"chunk32 {io}/{gate}/{precond}/{dk}x{dv}",
            chunk=32)


@pytest.mark.parametrize("T", [1, 16, 17, 31, 32, 33, 65, 100])
@pytest.mark.parametrize("gate", ["scalar", "channel"])
def test_bwd_chunk32_sequence_lengths(T, gate):
    """Last chunks of 1, 16 (one whole 16-token segment), 17 and 31 tokens,
    and whole chunks."""
    spec = pi.small_spec(T=T, B=1, H=2, gate=gate, dk=128, dv=128, with_do=True)
    compare(spec, pi.generate(spec, 600 + T), tag=f"chunk32 {gate} T={T}",
            chunk=32)


def test_bwd_chunk32_coverage():
    """beta in [0, 2], anisotropic keys, beta^P over decades, chunk = 32."""
    spec = pi.small_spec(gate="scalar", dk=128, dv=128, with_do=True,
                         beta_max=2.0, key_aniso=1.0, betap_logspan=2.0)
    compare(spec, pi.generate(spec, 31), tag="chunk32 beta02/aniso", chunk=32)
