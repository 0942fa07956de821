#!/usr/bin/env python
"""Throughput of the chunkwise preconditioned delta rule on one MI355X.

Default workload: the 1B-scale Preconditioned Gated DeltaNet layer (bf16 q/k/v,
fp32 state, B=4, T=4096, H=16, d_k=d_v=128, chunk 64, scalar gate, squash
preconditioner with x=1.5).  One step is one pass of the whole hot path over
the batch, with inputs resident in HBM: the forward (preconditioner scan,
per-chunk UT transform, inter-chunk state scan with the chunk output) and then
the backward for an upstream gradient dO (reverse state-adjoint scan,
per-chunk adjoint algebra, the preconditioner's reverse scan).  The step uses
the training pair: pdn_chunk_fwd_train leaves the forward intermediates in the
workspace and pdn_chunk_bwd_train reads them (--recompute times pdn_chunk_fwd
+ pdn_chunk_bwd, whose backward recomputes them).  --pass fwd times the
inference forward pdn_chunk_fwd alone.

Prints ONE JSON line: tokens/s (B*T per step time), the roofline of the
dominant kernel measured live with HIP events on the launch stream, and the
float64 CPU oracle (forward and adjoint) timed on a bounded sample on the
host's cores.
"""
from __future__ import annotations

import argparse
import dataclasses
import glob
import hashlib
import json
import re
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


def algorithmic_per_token_head(spec, train=False, precond="squash"):
    """Algorithmic FLOPs and bytes per token-head (one (b, t, h)).

    FLOPs: the dense per-chunk products as the paper writes them,
        forward  FLOP = 6 C dk + 4 C dv + 6 dk dv + C^2 / 3
        backward FLOP = 12 C dk + 8 C dv + 12 dk dv + 4 C^2
    (the backward's recompute of forward intermediates is executed work, not
    algorithmic, and is not in the totals).

    Bytes come in two kinds per kernel stage:
      method bytes  the method's own tensors the stage reads or writes, each
                    once: q, k, v, beta, g, betaP, gP (and the external write
                    key) in, o out; dO in, dq, dk, dv and the scalar
                    gradients out; the per-head states S0/S_T/A0/A_T and their
                    adjoints amortised over T.  Workspace intermediates are
                    not method bytes.  These define each stage's roofline
                    fraction.
      design bytes  what this design's stage must move as built: the method
                    bytes plus the intermediates it hands to other kernels
                    through HBM (solve factors, decayed keys, saved states,
                    E rows, state adjoints, ...), each once.
    Returns (flop_fwd, flop_bwd, {stage: (flop, method_bytes, design_bytes)},
    {"fwd": method bytes of a forward pass, "step": of the timed step}).
    """
    C, dk, dv = spec.chunk, spec.dk, spec.dv
    e = 2 if spec.io == "bf16" else 4
    gb = {"none": 0, "scalar": 4, "channel": 4 * dk}[spec.gate]
    gram = precond in ("squash", "diag_sm", "atq")
    pb = 8 if gram else 0                       # betaP, gP
    xk = e * dk if precond == "external" else 0  # external write key
    T = spec.T
    sh = 4 * dk * dv / T                         # one per-head state, per token
    ah = (4 * dk / T) if gram else 0.0           # one preconditioner state
    s0 = sh if spec.s0 != "zero" else 0.0        # S0 read
    st = e * dk * dv / C                         # one saved chunk-start state
    flop_fwd = 6 * C * dk + 4 * C * dv + 6 * dk * dv + C * C / 3.0
    flop_bwd = 12 * C * dk + 8 * C * dv + 12 * dk * dv + 4 * C * C
    # method bytes of whole passes
    fwd_in = e * (2 * dk + dv) + 4 + gb + pb + xk + s0 + ah   # A0 read
    fwd_m = fwd_in + e * dv + sh + ah                          # o, S_T, A_T
    bwd_m = (fwd_in + e * dv                                   # inputs, dO
             + e * (2 * dk + dv) + 4 + gb + pb + xk            # dq dk dv dbeta dg dbetaP dgP (dkt)
             + sh + ah)                                        # dS0, dA0
    # per stage: (flop, method bytes, design bytes)
    pre = (3 * dk, e * dk + pb + 2 * ah, e * dk + pb + 4 * dk / C)
    # k2: reads q, k, beta, g, betaP, gP and the chunk-start A; writes the
    # decayed write keys (dk), T and P (C each) and the gate prefix
    prep_m = e * 2 * dk + 4 + gb + pb + xk
    prep = (4 * C * dk + C * C / 3.0, prep_m,
            prep_m + 4 * dk / C + e * (dk + 2 * C) + gb)
    # k2 (backward mode): also P^T and M^T (C each) and the write-key,
    # decayed write-key, decayed query and key rows (dk each)
    prep_b = (prep[0], prep_m, prep[2] + 2 * e * C + 4 * e * dk)
    # k3: reads q, k, v; writes o and S_T (reads T, P, decayed write keys and
    # the gate prefix from the workspace)
    scan_m = e * (2 * dk + dv) + e * dv + s0 + sh
    scan = (6 * dk * dv + 4 * C * dv, scan_m,
            e * (2 * dk + dv) + e * (2 * C + dk) + gb + e * dv + s0 + sh)
    # k3 (saving, no output): reads k, v, T, decayed write keys, gate prefix;
    # writes the chunk-start states and the E rows
    save = (4 * dk * dv + 2 * C * dv, e * (dk + dv) + s0,
            e * (dk + dv) + e * (C + dk) + gb + st + e * dv + s0)
    if precond == "atq":
        # linear attention read through the preconditioned query: no
        # interaction matrix or solve; the prep kernel also writes the
        # preconditioned query rows, the scan reads them instead of q and k
        flop_fwd = 2 * C * dk + 2 * C * dv + 4 * dk * dv
        prep = (2 * C * dk, prep[1], prep[2] + e * dk)
        scan = (4 * dk * dv + 2 * C * dv, scan[1] - e * dk, scan[2] - e * dk)
    stages = {
        "precond": pre,
        "chunk_prep": prep_b if train else prep,
        # training forward: the output, the saved states and E rows
        "chunk_scan": ((scan[0], scan[1], scan[2] + st + e * dv) if train
                       else scan),
        "bwd_precond_recompute": pre,
        "bwd_chunk_prep": prep_b,
        "bwd_state_save_scan": save,
        # r1: reads dO and beta, writes dv and dS0 (method); also reads P^T,
        # M^T, the write keys, (lam Q)^T, -(lam K)^T and writes the state
        # adjoints and the Z rows
        "bwd_state_adjoint_scan": (4 * C * dv + 6 * dk * dv,
                                   2 * e * dv + 4 + sh,
                                   2 * e * C + 3 * e * dk + e * dv + 4
                                   + 4 / C + st + 2 * e * dv + sh),
        # p12: reads q, k, v, dO, beta, g; writes dq, dbeta, dg (method);
        # also reads Z, E, the write keys, the chunk-start states and their
        # adjoints and writes the key gradients of both keys
        "bwd_chunk_grads": (4 * C * dv + 12 * C * dk + 6 * dk * dv,
                            e * (2 * dk + 2 * dv) + 4 + gb + e * dk + 4 + gb,
                            4 * e * dv + 3 * e * dk + 2 * st + 4 + gb
                            + 3 * e * dk + 8),
        # pc: reads k, betaP, gP; writes dk, dbetaP, dgP, dA0 (method); also
        # reads both key gradients and the chunk-start A
        "bwd_precond_reverse": (10 * dk, e * dk + pb + e * dk + pb + ah,
                                3 * e * dk + 8 + 4 * dk / C + e * dk + 8),
    }
    return flop_fwd, flop_bwd, stages, {"fwd": fwd_m, "bwd": bwd_m}


SCAN_STAGES = ("chunk_scan", "bwd_state_save_scan", "bwd_state_adjoint_scan")

KERNELS = {
    "precond": "k1_precond_summary+k1_precond_carry",
    "chunk_prep": "k2_chunk_prep",
    "chunk_scan": "k3_chunk_scan",
    "chunk_prep_train": "k2_chunk_prep (backward mode)",
    "chunk_scan_train": "k3_chunk_scan (saving mode, with output)",
    "bwd_precond_recompute": "k1_precond_summary+k1_precond_carry",
    "bwd_chunk_prep": "k2_chunk_prep (backward mode)",
    "bwd_state_save_scan": "k3_chunk_scan (saving mode)",
    "bwd_state_adjoint_scan": "r1_state_adjoint",
    "bwd_chunk_grads": "p12_chunk_grads",
    "bwd_precond_reverse": "pc_chunk+pc_carry+pc_chunk+pc_mu",
}


def _oracle_job(args):
    from threadpoolctl import threadpool_limits
    from oracle import abi as oabi
    sample, kw, heads, bwd = args
    with threadpool_limits(1):
        t0 = time.perf_counter()
        oabi.forward(sample, heads=heads, **kw)
        if bwd:
            oabi.backward(sample, heads=heads, **kw)
        return time.perf_counter() - t0


def cpu_baseline(spec, inp, bwd, target_s=15.0, precond="squash", ridge=1.0,
                 knorm="none"):
    """Time the float64 oracle as it stands (token recurrence forward, and
    for bwd its adjoint as well) on a bounded sample: every head of the first
    nb batches over a prefix of Ts tokens, heads spread over worker
    processes.  nb and Ts are sized from a calibration run to about target_s
    of CPU time.  Returns the cpu_baseline object."""
    from concurrent.futures import ProcessPoolExecutor
    ncpu = len(os.sched_getaffinity(0))
    kw = dict(gate=spec.gate, precond=precond, x=spec.x, scale=spec.scale)
    if precond != "squash":
        kw["ridge"] = ridge
    if knorm != "none":
        kw["knorm"] = knorm

    def sample_of(nb, Ts):
        s = {}
        for key, a in inp.items():
            if a is None or (key == "dO" and not bwd):
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
        list(ex.map(_oracle_job, [(smp, kw, g, bwd) for g in groups]))
        return time.perf_counter() - t0, len(heads) * Ts

    # every core of the affinity set, unless the host declares a smaller CPU
    # share for this job through OMP_NUM_THREADS (the GPU hosts do: 16 per
    # GPU); never more workers than heads in the sample
    share = ncpu
    try:
        share = max(1, int(os.environ.get("OMP_NUM_THREADS", ncpu)))
    except ValueError:
        pass
    workers = max(1, min(ncpu, share, spec.B * spec.H))
    with ProcessPoolExecutor(max_workers=workers) as ex:
        run(ex, workers, 1, min(spec.T, 8))               # start the workers
        Tc = min(spec.T, 128)
        nbc = max(1, min(spec.B, -(-workers // spec.H)))
        tc, nc = run(ex, workers, nbc, Tc)
        rate = nc / tc                                     # token-heads / s
        want = rate * target_s
        nb = int(min(spec.B, max(1, round(want / (spec.H * spec.T)))))
        Ts = int(min(spec.T, max(Tc, want / (nb * spec.H))))
        wall, token_heads = run(ex, workers, nb, Ts)
    what = "forward + adjoint" if bwd else "forward"
    return {
        "value": (token_heads / spec.H) / wall,
        "unit": "tokens/s",
        "cores": workers,
        "kind": "oracle",
        "sample": (f"float64 token-recurrence oracle, {what}, batches "
                   f"0..{nb - 1} x all {spec.H} heads, first {Ts} of {spec.T} "
                   f"tokens ({token_heads} token-heads in {wall:.1f} s on "
                   f"{workers} worker processes x 1 thread; affinity set "
                   f"{ncpu} cores, declared CPU share {share}); value = "
                   f"token-heads/s / H"),
    }


def sources_sha256():
    """Hash of the HIP / host sources of the library (the kernels whose
    traffic a profile summary records)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2604_21100_amd", "csrc")
    for f in sorted(glob.glob(os.path.join(csrc, "*"))):
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode())
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload, mode, stage):
    """HBM bytes per launch of a stage's kernels, from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary of this workload (lines
    `traffic: <mode> <stage> <bytes>`), or None when there is none or the
    kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"sources-sha256: ([0-9a-f]{64})", text)
    if not m or m.group(1) != sources_sha256():
        return None
    m = re.search(rf"^traffic: {re.escape(mode)} {re.escape(stage)} (\d+)\s*$",
                  text, re.M)
    return int(m.group(1)) if m else None


def roofline_of(stage, ms, stages, token_heads, train=False, segs=1):
    """Roofline object for one kernel stage from its measured average time:
    `achieved` = the stage's method bytes (or FLOPs, when its method
    intensity is above the bf16 ridge) per launch / its time; the design's
    own compulsory bytes are reported beside it (design_bytes_per_launch,
    design_frac), and the counter traffic, when known, with its ratio to
    the method bytes.  When the scans are split along the sequence (`segs`
    > 1), a scan stage is two launches of its kernel with the segment
    composition between them, and its figures are per stage."""
    dflop, mbytes, dbytes = stages[stage]
    sec = ms / 1e3
    if dflop / mbytes >= PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9):
        ach = dflop * token_heads / sec / 1e12
        roof = {"bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s"}
    else:
        ach = mbytes * token_heads / sec / 1e9
        roof = {"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = None
    roof["kernel"] = KERNELS[stage + ("_train" if train and stage in
                                     ("chunk_prep", "chunk_scan") else "")]
    roof["stage"] = stage
    roof["launches_in_stage"] = 1
    if segs > 1 and stage in SCAN_STAGES:
        roof["kernel"] = (f"{roof['kernel']} x2 + seg_compose (sequence "
                          f"split into {segs} segments)")
        roof["launches_in_stage"] = 3
    roof["avg_ms"] = ms
    roof["alg_bytes_per_launch"] = mbytes * token_heads
    roof["alg_bytes_per_token_head"] = mbytes
    roof["alg_flop_per_launch"] = dflop * token_heads
    roof["mfma_frac"] = dflop * token_heads / sec / 1e12 / PEAK_BF16_TFLOPS
    roof["design_bytes_per_launch"] = dbytes * token_heads
    roof["design_frac"] = dbytes * token_heads / sec / 1e9 / PEAK_HBM_GBS
    return roof


def sweep(args):
    """Execution time against sequence length at batch 1, 8 heads, head
    dimension 128 (the kernel profiling setup of Sec. 5, efficiency
    analysis): for a scalar (PGDN) and a per-channel (PKDA) gate, each with
    the preconditioner (squash), with a given distinct write key and no
    preconditioner recurrence (external) and with the write key equal to the
    read key (identity: GDN / KDA).  Forward (pdn_chunk_fwd) and forward +
    backward (the training pair), HIP events around `steps` calls."""
    import torch
    import paper_2604_21100_amd as pdn
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    rows = []
    for T in [int(t) for t in args.sweep_t.split(",")]:
        for gate in ("scalar", "channel"):
            spec = pi.Spec(1, T, 8, 128, 128, gate=gate, with_do=True)
            inp = pi.generate(spec, 4000 + T)
            rng = np.random.default_rng(4100 + T)
            inp["ktilde"] = pi.round_bf16(
                inp["k"] * rng.uniform(1 / 1.5, 1.5, inp["k"].shape))
            d = {}
            for key, a in inp.items():
                if a is None:
                    d[key] = None
                    continue
                t = torch.from_numpy(np.ascontiguousarray(a))
                d[key] = (t.to(torch.bfloat16) if key in
                          ("q", "k", "v", "dO", "ktilde") else t).to(dev)
            for precond in ("squash", "external", "identity"):
                sq = precond == "squash"
                kw = dict(g=d["g"], gate=gate, precond=precond,
                          beta_p=d["beta_p"] if sq else None,
                          g_p=d["g_p"] if sq else None,
                          log_a_scale=d["log_a_scale"] if sq else None,
                          S0=d["S0"], x=spec.x, scale=spec.scale,
                          ktilde=d["ktilde"] if precond == "external" else None)
                prob = pdn.make_problem(1, T, 8, 128, 128, gate=gate,
                                        precond=precond)
                ws = torch.empty(pdn.pdn_workspace_size(prob, True),
                                 dtype=torch.uint8, device=dev)
                o = torch.empty_like(d["v"])
                grads = pdn.pdn_chunk_bwd(d["q"], d["k"], d["v"], d["beta"],
                                          d["dO"], workspace=ws, **kw)

                def fwd():
                    pdn.pdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], o=o,
                                      workspace=ws, stream=stream, **kw)

                def fwdbwd():
                    pdn.pdn_chunk_fwd(d["q"], d["k"], d["v"], d["beta"], o=o,
                                      workspace=ws, stream=stream, train=True,
                                      **kw)
                    pdn.pdn_chunk_bwd(d["q"], d["k"], d["v"], d["beta"],
                                      d["dO"], outputs=grads, workspace=ws,
                                      stream=stream, saved=True, **kw)

                def timed(fn):
                    for _ in range(args.warmup):
                        fn()
                    e0 = torch.cuda.Event(enable_timing=True)
                    e1 = torch.cuda.Event(enable_timing=True)
                    torch.cuda.synchronize()
                    e0.record(stream)
                    for _ in range(args.steps):
                        fn()
                    e1.record(stream)
                    torch.cuda.synchronize()
                    return e0.elapsed_time(e1) / args.steps

                row = {"T": T, "gate": gate, "precond": precond,
                       "fwd_ms": timed(fwd), "fwdbwd_ms": timed(fwdbwd)}
                row["fwd_tokens_per_s"] = T / (row["fwd_ms"] / 1e3)
                row["fwdbwd_tokens_per_s"] = T / (row["fwdbwd_ms"] / 1e3)
                rows.append(row)
                print(json.dumps(row), flush=True)
                del ws, grads
    print(f"{'T':>6} {'gate':8} {'precond':9} {'fwd ms':>8} {'fwd+bwd ms':>11}",
          file=sys.stderr)
    for r in rows:
        print(f"{r['T']:>6} {r['gate']:8} {r['precond']:9} {r['fwd_ms']:8.3f} "
              f"{r['fwdbwd_ms']:11.3f}", file=sys.stderr)
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD,
                    choices=sorted(pi.WORKLOADS))
    ap.add_argument("--pass", dest="passes", default="fwdbwd",
                    choices=("fwd", "fwdbwd"))
    ap.add_argument("--precond", default="squash",
                    choices=("squash", "diag_sm", "atq"),
                    help="write-key / query preconditioner: the method's "
                         "squash (default), the Sherman-Morrison write key "
                         "(diag_sm) or apply-to-query linear attention (atq); "
                         "the latter two are forward only")
    ap.add_argument("--ridge", type=float, default=0.1,
                    help="ridge lambda of diag_sm / atq")
    ap.add_argument("--knorm", default="none", choices=("none", "m", "1pm", "beta"),
                    help="normalisation factor on the squash write key (the "
                         "paper's ablation; forward only)")
    ap.add_argument("--recompute", action="store_true",
                    help="fwd+bwd with pdn_chunk_fwd + pdn_chunk_bwd (the "
                         "backward recomputes the forward intermediates)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--sweep", action="store_true",
                    help="kernel time against sequence length at B=1, H=8, "
                         "d=128 for the scalar and per-channel gates with "
                         "the preconditioner, with a given write key and "
                         "with k~ = k (one JSON line per point)")
    ap.add_argument("--sweep-t", default="1024,2048,4096,8192,16384,32768")
    ap.add_argument("--rotate", type=int, default=2,
                    help="input/output sets for the rotated (cold-MALL) "
                         "timing reported next to the hot one; 1 skips it")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also launch one device copy of this many MiB per "
                         "step (reference kernel for HBM counter scaling)")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py: one GPU only; --gpus {args.gpus} is not supported "
              "(sharding the (batch, head) pairs over several GPUs is not "
              "implemented)", file=sys.stderr)
        return 2

    if args.sweep:
        return sweep(args)
    bwd = args.passes == "fwdbwd"
    if bwd and (args.precond != "squash" or args.knorm != "none"):
        print(f"bench.py: --precond {args.precond} --knorm {args.knorm} is "
              "forward only; use --pass fwd", file=sys.stderr)
        return 2
    spec = pi.WORKLOADS[args.workload]
    if bwd and not spec.with_do:
        # dO is the last draw: every other input is unchanged
        spec = dataclasses.replace(spec, with_do=True)
    seed = pi.WORKLOAD_SEEDS[args.workload]
    inp = pi.generate(spec, seed)
    # the CPU leg runs before the GPU is touched (its worker processes fork)
    sq = args.precond == "squash"
    cpu = None if args.no_cpu_baseline else cpu_baseline(
        spec, inp, bwd, args.cpu_seconds, args.precond, args.ridge, args.knorm)

    import torch
    import paper_2604_21100_amd as pdn

    dev = torch.device("cuda:0")
    io_dt = torch.bfloat16 if spec.io == "bf16" else torch.float32
    d = {}
    for key, a in inp.items():
        if a is None:
            d[key] = None
            continue
        t = torch.from_numpy(np.ascontiguousarray(a))
        d[key] = (t.to(io_dt) if key in ("q", "k", "v", "dO") else t).to(dev)
    B, T, H, dk, dv = spec.B, spec.T, spec.H, spec.dk, spec.dv
    prob = pdn.make_problem(B, T, H, dk, dv, io=spec.io, gate=spec.gate,
                            precond=args.precond, x=spec.x, scale=spec.scale,
                            ridge=args.ridge, knorm=args.knorm)
    ws = torch.empty(pdn.pdn_workspace_size(prob, with_bwd=bwd),
                     dtype=torch.uint8, device=dev)

    def outputs():
        f32 = dict(dtype=torch.float32, device=dev)
        out = {"o": torch.empty((B, T, H, dv), dtype=io_dt, device=dev),
               "S_T": torch.empty((B, H, dk, dv), **f32),
               "A_T": torch.empty((B, H, dk), **f32), "grads": None}
        if bwd:
            out["grads"] = {
                "dq": torch.empty((B, T, H, dk), dtype=io_dt, device=dev),
                "dk": torch.empty((B, T, H, dk), dtype=io_dt, device=dev),
                "dv": torch.empty((B, T, H, dv), dtype=io_dt, device=dev),
                "dbeta": torch.empty((B, T, H), **f32),
                "dg": (torch.empty((B, T, H), **f32) if spec.gate == "scalar"
                       else torch.empty((B, T, H, dk), **f32)
                       if spec.gate == "channel" else None),
                "dS0": torch.empty((B, H, dk, dv), **f32),
                "dbeta_p": torch.empty((B, T, H), **f32),
                "dg_p": torch.empty((B, T, H), **f32),
                "dlog_a_scale": torch.empty((H,), **f32),
                "dA0": torch.empty((B, H, dk), **f32),
            }
        return out

    # set 0 is the hot-cache set; the rotated timing alternates it with
    # independent copies at other addresses (inputs and outputs), so that no
    # step finds its inputs in the 256 MB MALL the previous step left warm
    nrot = max(1, args.rotate)
    sets = [(d, outputs())]
    for _ in range(1, nrot):
        sets.append(({k: (None if v is None else v.clone()) for k, v in d.items()},
                     outputs()))
    calib = None
    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        calib = (torch.empty(n, dtype=torch.float32, device=dev).uniform_(),
                 torch.empty(n, dtype=torch.float32, device=dev))
    stream = torch.cuda.current_stream(dev)
    fwd_stages = list(pdn.FWD_STAGES)
    bwd_stages = list(pdn.BWD_STAGES) if bwd else []

    train = bwd and not args.recompute

    def step(fev=None, bev=None, which=0):
        x, out = sets[which]
        pdn.pdn_chunk_fwd(x["q"], x["k"], x["v"], x["beta"], g=x["g"],
                          gate=spec.gate, precond=args.precond,
                          beta_p=x["beta_p"], g_p=x["g_p"],
                          log_a_scale=x["log_a_scale"] if sq else None,
                          A0=x["A0"], S0=x["S0"], x=spec.x, scale=spec.scale,
                          ridge=args.ridge, knorm=args.knorm, o=out["o"],
                          S_T=out["S_T"], A_T=out["A_T"],
                          workspace=ws, stream=stream, stage_events=fev,
                          train=train)
        if bwd:
            pdn.pdn_chunk_bwd(x["q"], x["k"], x["v"], x["beta"], x["dO"],
                              g=x["g"], gate=spec.gate, beta_p=x["beta_p"],
                              g_p=x["g_p"], log_a_scale=x["log_a_scale"],
                              A0=x["A0"], S0=x["S0"], x=spec.x,
                              scale=spec.scale, outputs=out["grads"],
                              workspace=ws, stream=stream, stage_events=bev,
                              saved=train)
        if calib is not None:
            calib[1].copy_(calib[0])

    for _ in range(args.warmup):
        step()
    mk = lambda n: [torch.cuda.Event(enable_timing=True) for _ in range(n)]  # noqa: E731

    def stage_times(fev, bev, n):
        out = {}
        for si, name in enumerate(fwd_stages):
            if fev[0][si] is not None and fev[0][si + 1] is not None:
                out[name] = sum(fev[i][si].elapsed_time(fev[i][si + 1])
                                for i in range(n)) / n
        for si, name in enumerate(bwd_stages):
            if train and si < 3:
                continue   # the recompute stages are empty in the training pair
            if bev[0] is not None and bev[0][si] is not None and bev[0][si + 1] is not None:
                out[name] = sum(bev[i][si].elapsed_time(bev[i][si + 1])
                                for i in range(n)) / n
        return out

    # per-stage breakdown: a few untimed steps with an event at every stage
    # boundary (each record costs GPU time between kernels, so the timed
    # steps below record only the dominant stage's two boundaries)
    NC = 3
    cfev = [mk(len(fwd_stages) + 1) for _ in range(NC)]
    cbev = [mk(len(bwd_stages) + 1) for _ in range(NC)] if bwd else [None] * NC
    for i in range(NC):
        step(cfev[i], cbev[i])
    torch.cuda.synchronize()
    stage_ms = stage_times(cfev, cbev, NC)
    fwd_ms = sum(cfev[i][0].elapsed_time(cfev[i][-1]) for i in range(NC)) / NC
    bwd_ms = (sum(cbev[i][0].elapsed_time(cbev[i][-1]) for i in range(NC)) / NC
              if bwd else None)
    dom = max(stage_ms, key=stage_ms.get)

    K = args.steps

    def only_dom(names, stages_list, events):
        if dom not in stages_list:
            return [None] * (len(stages_list) + 1)
        si = stages_list.index(dom)
        return [events[j] if j in (si, si + 1) else None
                for j in range(len(stages_list) + 1)]

    def timed(rotate):
        """K steps between synchronisations, an event at every step
        boundary (for the median) and at the dominant stage's boundaries.
        Returns (total ms, per-step ms list, dominant stage ms, wall s)."""
        fev = [only_dom(fwd_stages, fwd_stages, mk(len(fwd_stages) + 1))
               for _ in range(K)]
        bev = ([only_dom(bwd_stages, bwd_stages, mk(len(bwd_stages) + 1))
                for _ in range(K)] if bwd else [None] * K)
        marks = mk(K + 1)
        torch.cuda.synchronize()
        t_wall = time.perf_counter()
        for i in range(K):
            marks[i].record(stream)
            step(fev[i], bev[i], i % nrot if rotate else 0)
        marks[K].record(stream)
        torch.cuda.synchronize()
        t_wall = time.perf_counter() - t_wall
        per = [marks[i].elapsed_time(marks[i + 1]) for i in range(K)]
        return (marks[0].elapsed_time(marks[K]), per,
                stage_times(fev, bev, K)[dom], t_wall)

    total_ms, per_step, dom_ms, t_wall = timed(False)
    ms_per_step = total_ms / K
    rot = None
    if nrot > 1:
        for i in range(nrot):          # touch every set once
            step(which=i)
        rtot, rper, rdom, _ = timed(True)
        rot = {"sets": nrot, "ms_per_step": rtot / K,
               "median_ms_per_step": float(np.median(rper)),
               "value": B * T / (rtot / K / 1e3),
               "dominant_stage_ms": rdom}

    tokens = B * T
    token_heads = B * T * H
    flop_fwd, flop_bwd, stages, passes = algorithmic_per_token_head(
        spec, train, args.precond)
    segs = pdn.pdn_scan_segments(prob)
    roof = roofline_of(dom, dom_ms, stages, token_heads, train, segs)
    mode = "train" if train else ("recompute" if bwd else "forward")
    roof["traffic"] = (measured_traffic(args.workload, mode, dom) if sq
                       else None)
    roof["traffic_over_alg"] = (None if roof["traffic"] is None else
                                roof["traffic"] / roof["alg_bytes_per_launch"])
    roof["traffic_over_design"] = (
        None if roof["traffic"] is None else
        roof["traffic"] / roof["design_bytes_per_launch"])
    if spec.gate == "channel":
        roof["kernel"] = roof["kernel"].replace("p12_", "p12c_")
    kernels = {}
    for k, v in stage_ms.items():
        r = roofline_of(k, v, stages, token_heads, train, segs)
        kernels[k] = {"frac": r["frac"], "design_frac": r["design_frac"],
                      "mfma_frac": r["mfma_frac"]}

    flop_step = flop_fwd + (flop_bwd if bwd else 0.0)
    step_s = ms_per_step / 1e3
    tflops = flop_step * token_heads / step_s / 1e12
    peak_tf = PEAK_BF16_TFLOPS if spec.io == "bf16" else PEAK_FP32_TFLOPS
    step_bytes = passes["fwd"] + (passes["bwd"] if bwd else 0.0)
    variant = {"scalar": "PGDN", "channel": "PKDA"}.get(spec.gate, "PDN")
    if args.precond == "atq":
        variant = {"scalar": "P-Mamba-2", "channel": "PGLA"}.get(spec.gate,
                                                                 "PLA")
    elif args.precond == "diag_sm":
        variant += " (Sherman-Morrison write key)"
    line = {
        "metric": "tokens/s of chunkwise PDN fwd(+bwd) at 1B layer shape; "
                  "% bf16 MFMA peak",
        "value": tokens / step_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "median_ms_per_step": float(np.median(per_step)),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.io,
        "data": "synthetic",
        "config": {"workload": args.workload, "variant": variant,
                   "pass": ("forward+backward (training pair)" if train
                            else "forward+backward (backward recomputes)"
                            if bwd else "forward"),
                   "B": B, "T": T, "H": H, "dk": dk, "dv": dv,
                   "chunk": spec.chunk, "gate": spec.gate,
                   "scan_segments": segs,
                   "precond": args.precond, "x": spec.x,
                   **({"ridge": args.ridge} if not sq else {}),
                   **({"knorm": args.knorm} if args.knorm != "none" else {}),
                   "global_batch": B,
                   "seq_len": T, "parallelism": "none (1 GPU)"},
        "tflops": tflops,
        "mfma_frac": tflops / peak_tf,
        "alg_flop_per_token_head": flop_step,
        "alg_bytes_per_token_head": step_bytes,
        "hbm_frac": step_bytes * token_heads / step_s / 1e9 / PEAK_HBM_GBS,
        "fwd_ms": fwd_ms,
        "fwd_tokens_per_s": tokens / (fwd_ms / 1e3),
        "bwd_ms": bwd_ms,
        "stage_ms": stage_ms,
        "stage_ms_source": (f"{NC} untimed steps with an event at every stage "
                            "boundary; fwd_ms / bwd_ms likewise; the timed "
                            "steps record only the dominant stage"),
        "stage_roofline": kernels,
        "wall_s_timed": t_wall,
        "rotated": rot,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
