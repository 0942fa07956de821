"""Seeded synthetic inputs for the chunkwise preconditioned delta rule.

This module is the only code shared by the CPU oracle and the HIP path: it
draws random tensors and rounds them to the storage precision the kernels
read.  It holds none of the method's arithmetic (no preconditioner, no
recurrence, no chunk algebra).

Distributions follow the paper's layer setup: unit-norm queries and keys
(the models L2-normalise q and k, App. E "Architectural hyperparameters"),
Gaussian values, a sigmoid write strength beta, log-decay gates
g = -0.1 * softplus(z) (scalar per token-head, or per key channel for the KDA
form), preconditioner gain beta^P = sigmoid(z) and decay g^P = -0.1*softplus(z)
(Eq. precond_end2end), logAScale = 0 (mu = 1) and x = 1.5 (App. E,
"Preconditioner hyperparameters").

Every array is returned in the C-ABI layout:
    q, k        [B, T, H, dk]      io values (float32 arrays holding bf16-exact
                                   values when io == "bf16")
    v, dO       [B, T, H, dv]      io values
    beta, g_p, beta_p  [B, T, H]   float32
    g           None | [B, T, H] | [B, T, H, dk]  float32
    log_a_scale [H]                float32
    S0          None | [B, H, dk, dv] float32  (the transpose of the paper's S)
    A0          None | [B, H, dk]  float32
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

__all__ = [
    "Spec", "WORKLOADS", "WORKLOAD_SEEDS", "round_bf16", "generate",
    "small_spec",
]


@dataclasses.dataclass(frozen=True)
class Spec:
    """Shape and distribution recipe of one synthetic problem."""
    B: int
    T: int
    H: int
    dk: int
    dv: int
    chunk: int = 64
    io: str = "bf16"            # "bf16" | "f32"
    gate: str = "none"          # "none" | "scalar" | "channel"
    s0: str = "zero"            # "zero" | "normal" (std 0.1)
    a0: str = "zero"            # "zero" | "lognormal"
    x: float = 1.5
    scale: float = 1.0
    with_do: bool = False
    # coverage knobs (untimed test inputs; they do not change shapes)
    beta_max: float = 1.0       # beta = beta_max * sigmoid(z); 2.0 for [0, 2]
    key_aniso: float = 0.0      # std of log-normal per-channel key scales
    betap_logspan: float = 0.0  # beta^P = sigmoid(z) * 10**U(-span, span)
    gate_strength: float = 0.1  # g = -gate_strength * softplus(z)
    log_a_scale: float = 0.0

    def replace(self, **kw) -> "Spec":
        return dataclasses.replace(self, **kw)


# The five layer workloads: names state variant, precision and sizes.
WORKLOADS = {
    # correctness-size PDN forward in fp32 (no gate)
    "pdn_fp32_b1_t256_h2_d64": Spec(1, 256, 2, 64, 64, io="f32"),
    # 340M-scale layer (D=1024, H=8, d=128, context 2048), PDN forward
    "pdn_bf16_b8_t2048_h8_d128": Spec(8, 2048, 8, 128, 128),
    # 1B-scale layer, PGDN forward, scalar gate
    "pgdn_bf16_b4_t4096_h16_d128": Spec(4, 4096, 16, 128, 128, gate="scalar"),
    # KDA-style layer, PKDA forward, per-channel gate, random initial state
    "pkda_bf16_b2_t8192_h16_d128": Spec(2, 8192, 16, 128, 128, gate="channel",
                                        s0="normal"),
    # long-context PGDN forward + backward with upstream dO ~ N(0, 1)
    "pgdn_fwdbwd_bf16_b1_t32768_h16_d128": Spec(1, 32768, 16, 128, 128,
                                                gate="scalar", with_do=True),
}
WORKLOAD_SEEDS = {name: 1001 + i for i, name in enumerate(WORKLOADS)}


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to bfloat16 (round to nearest, ties to even); returns float32."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    bias = np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))
    r = ((u + bias) >> np.uint64(16)) << np.uint64(16)
    return r.astype(np.uint32).view(np.float32).reshape(f.shape)


def _io(x: np.ndarray, io: str) -> np.ndarray:
    x = x.astype(np.float32)
    return round_bf16(x) if io == "bf16" else x


def _unit(z: np.ndarray) -> np.ndarray:
    return z / np.linalg.norm(z, axis=-1, keepdims=True)


def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def _softplus(z):
    return np.logaddexp(0.0, z)


def generate(spec: Spec, seed: int) -> dict:
    """Draw one problem.  Draw order is fixed: q, k, v, beta, g, beta^P,
    g^P, S0, dO, then the coverage knobs' extra draws."""
    rng = np.random.default_rng(seed)
    B, T, H, dk, dv = spec.B, spec.T, spec.H, spec.dk, spec.dv
    zq = rng.standard_normal((B, T, H, dk))
    zk = rng.standard_normal((B, T, H, dk))
    zv = rng.standard_normal((B, T, H, dv))
    zb = rng.standard_normal((B, T, H))
    if spec.gate == "scalar":
        zg = rng.standard_normal((B, T, H))
    elif spec.gate == "channel":
        zg = rng.standard_normal((B, T, H, dk))
    else:
        zg = None
    zbp = rng.standard_normal((B, T, H))
    zgp = rng.standard_normal((B, T, H))
    S0 = (0.1 * rng.standard_normal((B, H, dk, dv))).astype(np.float32) \
        if spec.s0 == "normal" else None
    dO = _io(rng.standard_normal((B, T, H, dv)), spec.io) if spec.with_do else None

    if spec.key_aniso > 0:
        ch = np.exp(spec.key_aniso * rng.standard_normal((1, 1, H, dk)))
        zk = zk * ch
    bp = _sigmoid(zbp)
    if spec.betap_logspan > 0:
        bp = bp * 10.0 ** rng.uniform(-spec.betap_logspan, spec.betap_logspan,
                                     size=bp.shape)
    A0 = None
    if spec.a0 == "lognormal":
        A0 = np.exp(rng.standard_normal((B, H, dk)) - 3.0).astype(np.float32)

    out = dict(
        q=_io(_unit(zq), spec.io),
        k=_io(_unit(zk), spec.io),
        v=_io(zv, spec.io),
        beta=(spec.beta_max * _sigmoid(zb)).astype(np.float32),
        g=None if zg is None else
        (-spec.gate_strength * _softplus(zg)).astype(np.float32),
        beta_p=bp.astype(np.float32),
        g_p=(-0.1 * _softplus(zgp)).astype(np.float32),
        log_a_scale=np.full((H,), spec.log_a_scale, dtype=np.float32),
        S0=S0,
        A0=A0,
        dO=dO,
    )
    return out


def small_spec(**kw) -> Spec:
    """A test-size problem: several chunks and a ragged tail by default."""
    base = dict(B=2, T=200, H=3, dk=64, dv=64, chunk=64, io="bf16",
                gate="scalar")
    base.update(kw)
    return Spec(**base)
