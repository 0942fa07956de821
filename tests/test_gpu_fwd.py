"""GPU parity of the forward pass (HIP kernels through the C ABI) against the
float64 oracle on the same seeded inputs.

Bar: max|x - r| / max|r| <= 1e-4 for fp32 io and <= 2e-2 for bf16 io (o and
S_T); the fp32 preconditioner state A_T is checked at 1e-4 in both cases.
Small problems are compared on every head; the full layer workloads on
sampled heads that the oracle computes one by one."""
import numpy as np
import pytest

import pdn_inputs as pi
from oracle import abi as oabi

from gpu_util import rel_err, run_fwd, tol

pytestmark = pytest.mark.gpu


def _oracle(spec, inp, precond="squash", heads=None, ridge=1.0):
    return oabi.forward(inp, gate=spec.gate, precond=precond, x=spec.x,
                        scale=spec.scale, heads=heads, B=spec.B, H=spec.H,
                        ridge=ridge)


def _check_all_heads(spec, inp, precond="squash", tag="", ridge=1.0):
    o, S_T, A_T = run_fwd(spec, inp, precond, ridge=ridge)
    ref = _oracle(spec, inp, precond, ridge=ridge)
    B, T, H = spec.B, spec.T, spec.H
    ro = np.stack([ref["o"][b * H + h] for b in range(B) for h in range(H)])
    go = np.stack([o[b, :, h] for b in range(B) for h in range(H)])
    e_o = rel_err(go, ro)
    e_s = rel_err(S_T.reshape(B * H, spec.dk, spec.dv), ref["S_T"])
    msg = f"{tag} err(o)={e_o:.2e} err(S_T)={e_s:.2e}"
    print(msg)
    assert e_o <= tol(spec.io), msg
    assert e_s <= tol(spec.io), msg
    if precond in ("squash", "diag_sm", "atq"):
        e_a = rel_err(A_T.reshape(B * H, spec.dk), ref["A_T"])
        assert e_a <= 1e-4, f"{tag} err(A_T)={e_a:.2e}"
    return o, S_T, A_T


SMALL = [
    # (io, gate, precond, dk, dv)
    ("bf16", "none", "squash", 128, 128),
    ("bf16", "scalar", "squash", 128, 128),
    ("bf16", "channel", "squash", 128, 128),
    ("bf16", "scalar", "identity", 128, 128),
    ("bf16", "channel", "identity", 64, 64),
    ("bf16", "none", "external", 128, 64),
    ("bf16", "scalar", "squash", 64, 128),
    ("f32", "none", "squash", 64, 64),
    ("f32", "scalar", "squash", 64, 64),
    ("f32", "channel", "squash", 64, 64),
    ("f32", "scalar", "identity", 128, 128),
    ("f32", "channel", "external", 128, 64),
]


@pytest.mark.parametrize("io,gate,precond,dk,dv", SMALL)
def test_small_all_heads(io, gate, precond, dk, dv):
    """Several chunks plus a ragged tail (T = 200 = 3*64 + 8), every head."""
    spec = pi.small_spec(io=io, gate=gate, dk=dk, dv=dv, s0="normal",
                         a0="lognormal" if precond == "squash" else "zero")
    inp = pi.generate(spec, 11)
    if precond == "external":
        rng = np.random.default_rng(5)
        kt = inp["k"] * rng.uniform(1 / 1.5, 1.5, inp["k"].shape)
        inp["ktilde"] = pi.round_bf16(kt) if io == "bf16" else kt.astype(np.float32)
    _check_all_heads(spec, inp, precond, tag=f"{io}/{gate}/{precond}/{dk}x{dv}")


MODES = [
    # (io, gate, precond, dk, dv, ridge): the Sherman-Morrison write key
    # (unstable ATK) and the apply-to-query linear attention (PLA /
    # P-Mamba-2 / PGLA), forward only
    ("bf16", "none", "diag_sm", 128, 128, 0.1),
    ("bf16", "scalar", "diag_sm", 128, 128, 0.1),
    ("bf16", "channel", "diag_sm", 64, 128, 0.5),
    ("f32", "scalar", "diag_sm", 64, 64, 0.1),
    ("f32", "channel", "diag_sm", 128, 64, 1.0),
    ("bf16", "none", "atq", 128, 128, 0.1),
    ("bf16", "scalar", "atq", 128, 128, 0.1),
    ("bf16", "channel", "atq", 128, 64, 0.5),
    ("f32", "channel", "atq", 64, 64, 0.1),
    ("f32", "none", "atq", 128, 128, 1.0),
]


@pytest.mark.parametrize("io,gate,precond,dk,dv,ridge", MODES)
def test_forward_only_modes(io, gate, precond, dk, dv, ridge):
    """T = 200 (ragged tail), every head, nonzero S0 and A0, beta^P and g^P
    as for the squash workloads."""
    spec = pi.small_spec(io=io, gate=gate, dk=dk, dv=dv, s0="normal",
                         a0="lognormal")
    inp = pi.generate(spec, 13)
    _check_all_heads(spec, inp, precond, ridge=ridge,
                     tag=f"{io}/{gate}/{precond}/{dk}x{dv}/ridge={ridge}")


KNORMS = [
    # (io, gate, knorm, dk, dv): the write-key normalisation ablation
    ("bf16", "scalar", "m", 128, 128),
    ("bf16", "none", "1pm", 128, 64),
    ("bf16", "scalar", "beta", 64, 128),
    ("bf16", "channel", "1pm", 128, 128),
    ("f32", "scalar", "beta", 64, 64),
    ("f32", "channel", "m", 64, 64),
]


@pytest.mark.parametrize("io,gate,knorm,dk,dv", KNORMS)
def test_squash_write_key_normalisations(io, gate, knorm, dk, dv):
    import torch
    spec = pi.small_spec(io=io, gate=gate, dk=dk, dv=dv, s0="normal",
                         a0="lognormal")
    inp = pi.generate(spec, 17)
    o, S_T, A_T = run_fwd(spec, inp, "squash", knorm=knorm)
    ref = oabi.forward(inp, gate=gate, precond="squash", x=spec.x,
                       scale=spec.scale, B=spec.B, H=spec.H, knorm=knorm)
    B, H = spec.B, spec.H
    go = np.stack([o[b, :, h] for b in range(B) for h in range(H)])
    e_o = rel_err(go, ref["o"])
    e_s = rel_err(S_T.reshape(B * H, dk, dv), ref["S_T"])
    msg = f"{io}/{gate}/knorm={knorm}/{dk}x{dv} err(o)={e_o:.2e} err(S_T)={e_s:.2e}"
    print(msg)
    assert e_o <= tol(io) and e_s <= tol(io), msg


@pytest.mark.parametrize("precond", ["diag_sm", "atq"])
@pytest.mark.parametrize("T", [1, 65, 129])
def test_forward_only_modes_lengths(precond, T):
    spec = pi.small_spec(T=T, B=1, H=2, gate="scalar", dk=128, dv=128)
    _check_all_heads(spec, pi.generate(spec, 700 + T), precond, ridge=0.2,
                     tag=f"{precond} T={T}")


@pytest.mark.parametrize("T", [1, 2, 63, 64, 65, 128, 129])
def test_sequence_lengths(T):
    spec = pi.small_spec(T=T, B=1, H=2, gate="scalar", dk=128, dv=128)
    _check_all_heads(spec, pi.generate(spec, 100 + T), tag=f"T={T}")


def test_empty_sequence_copies_states():
    import torch
    import paper_2604_21100_amd as pdn
    spec = pi.small_spec(T=0, B=2, H=2, s0="normal", a0="lognormal")
    inp = pi.generate(spec, 3)
    from gpu_util import to_device
    d = to_device(inp, "bf16")
    o, S_T, A_T = pdn.pdn_chunk_fwd(
        d["q"], d["k"], d["v"], d["beta"], g=d["g"], gate="scalar",
        beta_p=d["beta_p"], g_p=d["g_p"], log_a_scale=d["log_a_scale"],
        A0=d["A0"], S0=d["S0"])
    torch.cuda.synchronize()
    assert o.numel() == 0
    assert np.array_equal(S_T.cpu().numpy(), inp["S0"])
    assert np.array_equal(A_T.cpu().numpy(), inp["A0"])


@pytest.mark.parametrize("case", ["beta_0_2", "squash_coverage", "x_2",
                                  "x_1", "scale", "strong_gate", "strong_channel_gate",
                                  "zero_key_channel", "no_gp"])
def test_edge_cases(case):
    kw = dict(gate="scalar", dk=128, dv=128)
    if case == "beta_0_2":
        kw.update(beta_max=2.0)                    # negative eigenvalues, no clamping
    if case == "squash_coverage":
        kw.update(key_aniso=1.5, betap_logspan=4.0)  # B on both sides of 1
    if case == "x_2":
        kw.update(x=2.0)
    if case == "x_1":
        kw.update(x=1.0)
    if case == "scale":
        kw.update(scale=0.0883883)
    if case == "strong_gate":
        kw.update(gate_strength=3.0)
    if case == "strong_channel_gate":
        kw.update(gate="channel", gate_strength=1.5)
    spec = pi.small_spec(**kw)
    inp = pi.generate(spec, 7)
    if case == "zero_key_channel":
        inp["k"][:, :, :, 5] = 0.0                 # A = 0 limit: B = x
    if case == "no_gp":
        inp["g_p"] = None
    _check_all_heads(spec, inp, tag=case)


def test_x1_squash_equals_identity():
    """x = 1 makes the write key equal the read key exactly (B = 1)."""
    spec = pi.small_spec(x=1.0, gate="channel")
    inp = pi.generate(spec, 9)
    a = run_fwd(spec, inp, "squash")
    b = run_fwd(spec, inp, "identity")
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_deterministic():
    spec = pi.small_spec(B=3, H=5, T=333, gate="channel", s0="normal")
    inp = pi.generate(spec, 13)
    a = run_fwd(spec, inp)
    b = run_fwd(spec, inp)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_split_sequence_chaining():
    """(S_T, A_T) of a first call fed as (S0, A0) of a second call on the
    rest of the sequence reproduces the oracle over the whole sequence."""
    spec = pi.small_spec(B=2, H=2, T=300, gate="scalar")
    inp = pi.generate(spec, 17)
    tau = 100
    first = {k: (None if v is None else (v[:, :tau] if v.ndim >= 3 else v))
             for k, v in inp.items()}
    for key in ("log_a_scale", "S0", "A0"):
        first[key] = inp[key]
    o1, S1, A1 = run_fwd(spec.replace(T=tau), first)
    second = {k: (None if v is None else (v[:, tau:] if v.ndim >= 3 else v))
              for k, v in inp.items()}
    second["log_a_scale"] = inp["log_a_scale"]
    second["S0"] = S1.astype(np.float32)
    second["A0"] = A1.astype(np.float32)
    o2, S2, A2 = run_fwd(spec.replace(T=spec.T - tau), second)
    ref = _oracle(spec, inp)
    o = np.concatenate([o1, o2], axis=1)
    ro = np.stack([ref["o"][b * 2 + h] for b in range(2) for h in range(2)])
    go = np.stack([o[b, :, h] for b in range(2) for h in range(2)])
    assert rel_err(go, ro) <= 2e-2
    assert rel_err(S2.reshape(4, spec.dk, spec.dv), ref["S_T"]) <= 2e-2
    assert rel_err(A2.reshape(4, spec.dk), ref["A_T"]) <= 1e-4


FULL = ["pdn_fp32_b1_t256_h2_d64", "pdn_bf16_b8_t2048_h8_d128",
        "pgdn_bf16_b4_t4096_h16_d128", "pkda_bf16_b2_t8192_h16_d128",
        "pgdn_fwdbwd_bf16_b1_t32768_h16_d128"]


@pytest.mark.parametrize("name", FULL)
def test_full_workload_sampled_heads(name):
    """Full-size layer workloads in the benchmark's launch configuration;
    the oracle recomputes two sampled heads (first and last) end to end."""
    spec = pi.WORKLOADS[name]
    inp = pi.generate(spec, pi.WORKLOAD_SEEDS[name])
    o, S_T, A_T = run_fwd(spec, inp)
    heads = [(0, 0), (spec.B - 1, spec.H - 1)]
    ref = _oracle(spec, inp, heads=heads)
    for n, (b, h) in enumerate(heads):
        e_o = rel_err(o[b, :, h], ref["o"][n])
        e_s = rel_err(S_T[b, h], ref["S_T"][n])
        e_a = rel_err(A_T[b, h], ref["A_T"][n])
        print(f"{name} head {(b, h)}: err(o)={e_o:.2e} err(S_T)={e_s:.2e} err(A_T)={e_a:.2e}")
        assert e_o <= tol(spec.io) and e_s <= tol(spec.io) and e_a <= 1e-4
    assert np.isfinite(o).all() and np.isfinite(S_T).all()


@pytest.mark.parametrize("precond,gate,ridge", [("diag_sm", "scalar", 0.1),
                                                ("atq", "scalar", 0.1),
                                                ("atq", "channel", 0.1)])
def test_forward_only_modes_full_layer(precond, gate, ridge):
    """The forward-only modes at the 1B layer shape (B=4, T=4096, H=16,
    d=128; the PGLA case with the PKDA layer's per-channel gate recipe) in
    the benchmark's launch configuration; two sampled heads end to end."""
    name = "pgdn_bf16_b4_t4096_h16_d128"
    spec = pi.WORKLOADS[name].replace(gate=gate)
    inp = pi.generate(spec, pi.WORKLOAD_SEEDS[name])
    o, S_T, A_T = run_fwd(spec, inp, precond, ridge=ridge)
    heads = [(0, 0), (spec.B - 1, spec.H - 1)]
    ref = _oracle(spec, inp, precond, heads=heads, ridge=ridge)
    for n, (b, h) in enumerate(heads):
        e_o = rel_err(o[b, :, h], ref["o"][n])
        e_s = rel_err(S_T[b, h], ref["S_T"][n])
        e_a = rel_err(A_T[b, h], ref["A_T"][n])
        print(f"{precond}/{gate} head {(b, h)}: err(o)={e_o:.2e} err(S_T)={e_s:.2e} err(A_T)={e_a:.2e}")
        assert e_o <= tol(spec.io) and e_s <= tol(spec.io) and e_a <= 1e-4


CHUNK32 = [
    # (io, gate, precond, dk, dv, ridge): 32-token chunks (two 16-row blocks
    # per chunk) across gates, write keys and the forward-only modes
    ("bf16", "none", "squash", 128, 128, 1.0),
    ("bf16", "scalar", "squash", 128, 128, 1.0),
    ("bf16", "channel", "squash", 128, 128, 1.0),
    ("bf16", "scalar", "identity", 64, 128, 1.0),
    ("bf16", "channel", "external", 128, 64, 1.0),
    ("f32", "scalar", "squash", 64, 64, 1.0),
    ("f32", "channel", "identity", 64, 64, 1.0),
    ("f32", "none", "squash", 128, 128, 1.0),
    ("bf16", "scalar", "diag_sm", 128, 128, 0.1),
    ("bf16", "channel", "atq", 128, 64, 0.5),
    ("f32", "scalar", "atq", 64, 64, 0.1),
]


@pytest.mark.parametrize("io,gate,precond,dk,dv,ridge", CHUNK32)
def test_chunk32_all_heads(io, gate, precond, dk, dv, ridge):
    """chunk = 32: T = 200 = 6*32 + 8 (ragged tail), every head, nonzero S0
    and A0, against the token recurrence (which has no chunk)."""
    spec = pi.small_spec(io=io, gate=gate, dk=dk, dv=dv, s0="normal",
                         a0="lognormal" if precond != "identity" and
                         precond != "external" else "zero")
    inp = pi.generate(spec, 19)
    if precond == "external":
        rng = np.random.default_rng(5)
        kt = inp["k"] * rng.uniform(1 / 1.5, 1.5, inp["k"].shape)
        inp["ktilde"] = pi.round_bf16(kt) if io == "bf16" else kt.astype(np.float32)
    o, S_T, A_T = run_fwd(spec, inp, precond, ridge=ridge, chunk=32)
    ref = _oracle(spec, inp, precond, ridge=ridge)
    B, H = spec.B, spec.H
    go = np.stack([o[b, :, h] for b in range(B) for h in range(H)])
    e_o = rel_err(go, ref["o"])
    e_s = rel_err(S_T.reshape(B * H, dk, dv), ref["S_T"])
    msg = f"chunk32 {io}/{gate}/{precond}/{dk}x{dv} err(o)={e_o:.2e} err(S_T)={e_s:.2e}"
    print(msg)
    assert e_o <= tol(io) and e_s <= tol(io), msg
    if A_T is not None:
        assert rel_err(A_T.reshape(B * H, dk), ref["A_T"]) <= 1e-4


@pytest.mark.parametrize("T", [1, 31, 32, 33, 64, 95, 97])
@pytest.mark.parametrize("gate", ["scalar", "channel"])
def test_chunk32_sequence_lengths(T, gate):
    spec = pi.small_spec(T=T, B=1, H=2, gate=gate, dk=128, dv=128, s0="normal")
    inp = pi.generate(spec, 900 + T)
    o, S_T, A_T = run_fwd(spec, inp, chunk=32)
    ref = _oracle(spec, inp)
    go = np.stack([o[0, :, h] for h in range(2)])
    e_o, e_s = rel_err(go, ref["o"]), rel_err(S_T.reshape(2, 128, 128), ref["S_T"])
    print(f"chunk32 {gate} T={T} err(o)={e_o:.2e} err(S_T)={e_s:.2e}")
    assert e_o <= 2e-2 and e_s <= 2e-2
    assert rel_err(A_T.reshape(2, 128), ref["A_T"]) <= 1e-4


def test_chunk32_full_layer_sampled_heads():
    """The 1B PGDN layer (B=4, T=4096, H=16, d=128) with 32-token chunks:
    two sampled heads against the oracle, and the result close to the
    64-token chunking of the same inputs."""
    name = "pgdn_bf16_b4_t4096_h16_d128"
    spec = pi.WORKLOADS[name]
    inp = pi.generate(spec, pi.WORKLOAD_SEEDS[name])
    o, S_T, A_T = run_fwd(spec, inp, chunk=32)
    heads = [(0, 0), (spec.B - 1, spec.H - 1)]
    ref = _oracle(spec, inp, heads=heads)
    for n, (b, h) in enumerate(heads):
        e_o = rel_err(o[b, :, h], ref["o"][n])
        e_s = rel_err(S_T[b, h], ref["S_T"][n])
        print(f"chunk32 {name} head {(b, h)}: err(o)={e_o:.2e} err(S_T)={e_s:.2e}")
        assert e_o <= 2e-2 and e_s <= 2e-2
        assert rel_err(A_T[b, h], ref["A_T"][n]) <= 1e-4
    o64, S64, _ = run_fwd(spec, inp, chunk=64)
    assert rel_err(o, o64) <= 2e-2 and rel_err(S_T, S64) <= 2e-2
