#!/usr/bin/env python
"""Throughput of the chunkwise preconditioned delta rule on one MI355X.

Default workload: the 1B-scale Preconditioned Gated DeltaNet layer (bf16 q/k/v,
fp32 state, B=4, T=4096, H=16, d_k=d_v=128, chunk 64, scalar gate, squash
preconditioner with x=1.5).  One step is one pass of the forward hot path
(preconditioner scan, per-chunk UT transform, inter-chunk state scan with the
chunk output) over the whole batch, with inputs resident in HBM.

Prints ONE JSON line: tokens/s (B*T per step time), the roofline of the
dominant kernel measured live with HIP events on the launch stream, and the
float64 CPU oracle timed on a bounded sample on the host's cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import pdn_inputs as pi  # noqa: E402

DEFAULT_WORKLOAD = "pgdn_bf16_b4_t4096_h16_d128"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0      # dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3       # dense fp32 matrix


def algorithmic_per_token_head(spec):
    """Algorithmic FLOPs and bytes per token-head (one (b, t, h)).

    Whole forward (dense per-chunk products as the paper writes them):
        FLOP = 6 C dk + 4 C dv + 6 dk dv + C^2 / 3
    and the compulsory bytes of each kernel (inputs read once, outputs written
    once).  Returns (flop_total, {stage: (flop, bytes)})."""
    C, dk, dv = spec.chunk, spec.dk, spec.dv
    e = 2 if spec.io == "bf16" else 4
    gate_b = {"none": 0, "scalar": 4, "channel": 4 * dk}[spec.gate]
    flop = 6 * C * dk + 4 * C * dv + 6 * dk * dv + C * C / 3.0
    stages = {
        # k1: read k, betaP, gP; write the per-chunk summaries
        "precond": (3 * dk, e * dk + 8 + 4 * dk / C),
        # k2: read q, k, beta, g, betaP, gP, chunk-start A; write the decayed
        # write keys (dk), T and P (C each) and the gate prefix
        "chunk_prep": (4 * C * dk + C * C / 3.0,
                       2 * e * dk + 12 + gate_b + 4 * dk / C
                       + e * (dk + 2 * C) + gate_b),
        # k3: read q, k, v, T, P, decayed write keys, gate prefix; write o
        "chunk_scan": (6 * dk * dv + 4 * C * dv,
                       e * (2 * dk + dv) + e * (2 * C + dk) + gate_b + e * dv),
    }
    return flop, stages


def _oracle_job(args):
    from threadpoolctl import threadpool_limits
    from oracle import abi as oabi
    sample, kw, heads = args
    with threadpool_limits(1):
        t0 = time.perf_counter()
        oabi.forward(sample, heads=heads, **kw)
        return time.perf_counter() - t0


def cpu_baseline(spec, inp, target_s=15.0):
    """Time the float64 oracle (token recurrence, as it stands) on a bounded
    sample: every head of the first nb batches over a prefix of Ts tokens,
    heads spread over worker processes.  nb and Ts are sized from a
    calibration run to about target_s of CPU time.  Returns the cpu_baseline
    object."""
    from concurrent.futures import ProcessPoolExecutor
    ncpu = len(os.sched_getaffinity(0))
    kw = dict(gate=spec.gate, precond="squash", x=spec.x, scale=spec.scale)

    def sample_of(nb, Ts):
        s = {}
        for key, a in inp.items():
            if a is None or key == "dO":
                s[key] = None
            elif key == "log_a_scale":
                s[key] = a
            elif key in ("S0", "A0"):
                s[key] = a[:nb]
            else:
                s[key] = a[:nb, :Ts]
        return s

    def run(ex, workers, nb, Ts):
        heads = [(b, h) for b in range(nb) for h in range(spec.H)]
        groups = [g for g in (heads[i::workers] for i in range(workers)) if g]
        smp = sample_of(nb, Ts)
        t0 = time.perf_counter()
        list(ex.map(_oracle_job, [(smp, kw, g) for g in groups]))
        return time.perf_counter() - t0, len(heads) * Ts

    workers = max(1, min(16, ncpu, spec.B * spec.H))
    with ProcessPoolExecutor(max_workers=workers) as ex:
        run(ex, workers, 1, min(spec.T, 8))               # start the workers
        Tc = min(spec.T, 256)
        nbc = max(1, min(spec.B, -(-workers // spec.H)))
        tc, nc = run(ex, workers, nbc, Tc)
        rate = nc / tc                                     # token-heads / s
        want = rate * target_s
        nb = int(min(spec.B, max(1, round(want / (spec.H * spec.T)))))
        Ts = int(min(spec.T, max(Tc, want / (nb * spec.H))))
        wall, token_heads = run(ex, workers, nb, Ts)
    return {
        "value": (token_heads / spec.H) / wall,
        "unit": "tokens/s",
        "cores": workers,
        "kind": "oracle",
        "sample": (f"float64 token-recurrence oracle, forward, batches 0..{nb - 1}"
                   f" x all {spec.H} heads, first {Ts} of {spec.T} tokens "
                   f"({token_heads} token-heads in {wall:.1f} s on {workers} "
                   f"worker processes x 1 thread); value = token-heads/s / H"),
    }


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD,
                    choices=sorted(pi.WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also launch one device copy of this many MiB per "
                         "step (reference kernel for HBM counter scaling)")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is "
              "not supported (the (b, h) sharding across GPUs is described "
              "in DESIGN.md but not built)", file=sys.stderr)
        return 2

    spec = pi.WORKLOADS[args.workload]
    seed = pi.WORKLOAD_SEEDS[args.workload]
    inp = pi.generate(spec, seed)
    # the CPU leg runs before the GPU is touched (its worker processes fork)
    cpu = None if args.no_cpu_baseline else cpu_baseline(spec, inp,
                                                         args.cpu_seconds)

    import torch
    import paper_2604_21100_amd as pdn

    dev = torch.device("cuda:0")
    io_dt = torch.bfloat16 if spec.io == "bf16" else torch.float32
    d = {}
    for key, a in inp.items():
        if a is None or key == "dO":
            d[key] = None
            continue
        t = torch.from_numpy(np.ascontiguousarray(a))
        d[key] = (t.to(io_dt) if key in ("q", "k", "v") else t).to(dev)
    B, T, H, dk, dv = spec.B, spec.T, spec.H, spec.dk, spec.dv
    o = torch.empty((B, T, H, dv), dtype=io_dt, device=dev)
    S_T = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev)
    A_T = torch.empty((B, H, dk), dtype=torch.float32, device=dev)
    prob = pdn.make_problem(B, T, H, dk, dv, io=spec.io, gate=spec.gate,
                            x=spec.x, scale=spec.scale)
    ws = torch.empty(pdn.pdn_workspace_size(prob), dtype=torch.uint8,
                     device=dev)
    calib = None
    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        calib = (torch.empty(n, dtype=torch.float32, device=dev).uniform_(),
                 torch.empty(n, dtype=torch.float32, device=dev))
    stream = torch.cuda.current_stream(dev)

    def step(events=None):
        pdn.pdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], g=d["g"],
                          gate=spec.gate, beta_p=d["beta_p"], g_p=d["g_p"],
                          log_a_scale=d["log_a_scale"], A0=d["A0"],
                          S0=d["S0"], x=spec.x, scale=spec.scale, o=o,
                          S_T=S_T, A_T=A_T, workspace=ws, stream=stream,
                          stage_events=events)
        if calib is not None:
            calib[1].copy_(calib[0])

    for _ in range(args.warmup):
        step()
    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)]
          for _ in range(K)]
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record(stream)
    for i in range(K):
        step(ev[i])
    end.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / K
    stage_ms = {}
    for si, name in enumerate(pdn.FWD_STAGES):
        stage_ms[name] = sum(ev[i][si].elapsed_time(ev[i][si + 1])
                             for i in range(K)) / K

    tokens = B * T
    token_heads = B * T * H
    flop_tok, stages = algorithmic_per_token_head(spec)
    dom = max(stage_ms, key=stage_ms.get)
    dflop, dbytes = stages[dom]
    dom_s = stage_ms[dom] / 1e3
    if dflop / dbytes >= PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9):
        ach = dflop * token_heads / dom_s / 1e12
        roof = {"bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s"}
    else:
        ach = dbytes * token_heads / dom_s / 1e9
        roof = {"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = None
    roof["kernel"] = {"precond": "k1_precond_summary+k1_precond_carry",
                      "chunk_prep": "k2_chunk_prep",
                      "chunk_scan": "k3_chunk_scan"}[dom]
    roof["avg_ms"] = stage_ms[dom]
    roof["alg_bytes_per_launch"] = dbytes * token_heads
    roof["alg_flop_per_launch"] = dflop * token_heads

    step_s = ms_per_step / 1e3
    tflops = flop_tok * token_heads / step_s / 1e12
    peak_tf = PEAK_BF16_TFLOPS if spec.io == "bf16" else PEAK_FP32_TFLOPS
    line = {
        "metric": "tokens/s of chunkwise PDN fwd(+bwd) at 1B layer shape; "
                  "% bf16 MFMA peak",
        "value": tokens / step_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.io,
        "data": "synthetic",
        "config": {"workload": args.workload, "variant": "PGDN" if spec.gate == "scalar" else ("PKDA" if spec.gate == "channel" else "PDN"),
                   "pass": "forward", "B": B, "T": T, "H": H, "dk": dk,
                   "dv": dv, "chunk": spec.chunk, "gate": spec.gate,
                   "precond": "squash", "x": spec.x, "global_batch": B,
                   "seq_len": T, "parallelism": "none (1 GPU)"},
        "tflops": tflops,
        "mfma_frac": tflops / peak_tf,
        "alg_flop_per_token_head": flop_tok,
        "stage_ms": stage_ms,
        "wall_s_timed": t_wall,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
