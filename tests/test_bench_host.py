"""Host-side checks of bench.py's accounting (no GPU): the per-token-head
method bytes it prices rooflines with, the roofline object of a stage
(including a scan stage split along the sequence), the counter-traffic
lookup keyed by the kernel sources' hash, and the one-GPU guard."""
import pytest

import bench
import pdn_inputs as pi


def _spec():
    return pi.WORKLOADS[bench.DEFAULT_WORKLOAD]


def test_method_bytes_of_the_training_step():
    # bf16 B=4 T=4096 H=16 d=128: the chunk-gradient stage reads q, k, v,
    # dO, beta, g and writes dq, dk, dv, dbeta, dg (each once), 1,296 B a
    # token-head; the whole training step 2,896 B
    ff, fb, stages, passes = bench.algorithmic_per_token_head(_spec(), True)
    dflop, mbytes, dbytes = stages["bwd_chunk_grads"]
    assert mbytes == pytest.approx(1296, abs=1)
    assert dbytes > mbytes
    assert passes["fwd"] + passes["bwd"] == pytest.approx(2896, abs=1)
    assert ff > 0 and fb > ff


def test_roofline_fields_and_split_stage():
    spec = _spec()
    ff, fb, stages, _ = bench.algorithmic_per_token_head(spec, True)
    th = spec.B * spec.T * spec.H
    r = bench.roofline_of("bwd_chunk_grads", 0.25, stages, th, True)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s"
    assert r["frac"] == pytest.approx(r["achieved"] / r["peak"])
    assert r["achieved"] == pytest.approx(r["alg_bytes_per_launch"] / 0.25e-3 / 1e9)
    assert r["launches_in_stage"] == 1 and "seg_compose" not in r["kernel"]
    s = bench.roofline_of("bwd_state_adjoint_scan", 1.0, stages, th, True, segs=3)
    assert s["launches_in_stage"] == 3
    assert s["kernel"].startswith("r1_state_adjoint x2 + seg_compose")
    # a stage that is never split keeps one launch
    p = bench.roofline_of("bwd_chunk_grads", 0.25, stages, th, True, segs=3)
    assert p["launches_in_stage"] == 1


def test_traffic_lookup_is_keyed_by_the_sources():
    # a committed summary is used only while its recorded hash is that of the
    # current kernel sources; a workload without a summary has no traffic
    import os
    import re
    path = os.path.join(bench.ROOT, "profiles", f"traffic_{bench.DEFAULT_WORKLOAD}.md")
    m = re.search(r"sources-sha256: ([0-9a-f]{64})", open(path).read())
    fresh = m is not None and m.group(1) == bench.sources_sha256()
    t = bench.measured_traffic(bench.DEFAULT_WORKLOAD, "train", "bwd_chunk_grads")
    assert (t is not None) == fresh
    if fresh:
        assert t > 0
    assert bench.measured_traffic("pkda_bf16_b2_t8192_h16_d128", "train", "bwd_chunk_grads") is None


def test_more_than_one_gpu_is_refused():
    assert bench.main(["--gpus", "2"]) == 2
