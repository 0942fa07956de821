"""The seeded input generator: shapes, determinism, storage rounding."""
import numpy as np

import pdn_inputs as pi


def test_round_bf16_ties_to_even_and_exactness():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9,
                  -2.5, 3.140625], dtype=np.float32)
    r = pi.round_bf16(x)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: rounds to even (1.0)
    assert r[1] == 1.0 and r[2] == 1.0 + 2 ** -6 and r[3] == 1.0
    assert r[4] == -2.5 and r[5] == 3.140625
    assert np.array_equal(pi.round_bf16(r), r)


def test_generate_shapes_and_determinism():
    s = pi.small_spec(gate="channel", s0="normal", with_do=True)
    a = pi.generate(s, 5)
    b = pi.generate(s, 5)
    for key in a:
        if a[key] is None:
            assert b[key] is None
        else:
            assert np.array_equal(a[key], b[key])
    assert a["q"].shape == (2, 200, 3, 64) and a["g"].shape == (2, 200, 3, 64)
    assert a["S0"].shape == (2, 3, 64, 64) and a["dO"].shape == (2, 200, 3, 64)
    assert np.array_equal(pi.round_bf16(a["k"]), a["k"])
    n = np.linalg.norm(a["k"].astype(np.float64), axis=-1)
    assert np.abs(n - 1).max() < 1e-2
    assert (a["g"] < 0).all() and (a["beta"] > 0).all() and (a["beta"] < 1).all()


def test_workload_table():
    assert set(pi.WORKLOADS) == set(pi.WORKLOAD_SEEDS)
    w = pi.WORKLOADS["pgdn_bf16_b4_t4096_h16_d128"]
    assert (w.B, w.T, w.H, w.dk, w.dv, w.chunk, w.gate) == (4, 4096, 16, 128,
                                                           128, 64, "scalar")
