"""Pins for the float64 oracle: each test checks the oracle against something
other than itself -- a value the paper prints, a closed form, an invariant
the paper proves, a library routine, or finite differences.  CPU only."""
import os

import numpy as np
import pytest

from oracle import adjoint, chunkwise, lsq, recurrent

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _unit(z):
    return z / np.linalg.norm(z, axis=-1, keepdims=True)


def _sig(z):
    return 1.0 / (1.0 + np.exp(-z))


def _rand_problem(rng, N, T, dk, dv, gate):
    q = _unit(rng.standard_normal((N, T, dk)))
    k = _unit(rng.standard_normal((N, T, dk)))
    v = rng.standard_normal((N, T, dv))
    beta = _sig(rng.standard_normal((N, T)))
    g = None
    if gate == "scalar":
        g = -0.1 * np.logaddexp(0, rng.standard_normal((N, T)))
    elif gate == "channel":
        g = -0.1 * np.logaddexp(0, rng.standard_normal((N, T, dk)))
    bp = _sig(rng.standard_normal((N, T)))
    gp = -0.1 * np.logaddexp(0, rng.standard_normal((N, T)))
    mu = np.exp(0.3 * rng.standard_normal(N))
    return q, k, v, beta, g, bp, gp, mu


# ---------------------------------------------------------------- Sec. 3.1
@pytest.mark.parametrize("dk,dv,T,lam", [(2, 2, 6, 1.0), (4, 3, 12, 0.1),
                                         (8, 5, 32, 1.0), (3, 4, 10, 0.1)])
def test_exact_gram_pdn_is_ridge_least_squares(dk, dv, T, lam):
    """Theorem (PDN == PLA == least squares under the exact inverse Gram):
    S_t equals the ridge least-squares map at every t; kt_t = P_t k_t; and
    the outputs equal the apply-to-query read-out C_t (P_t q_t)."""
    rng = np.random.default_rng(dk * 100 + T)
    K = rng.standard_normal((T, dk))
    V = rng.standard_normal((T, dv))
    Q = rng.standard_normal((T, dk))
    S_all, kts, P_all, o = recurrent.exact_gram_pdn(K, V, Q, lam)
    L = lsq.ridge_maps(K, V, lam)
    assert np.abs(S_all - L).max() <= 1e-10 * max(1.0, np.abs(L).max())
    for t in range(T):
        G = K[:t + 1].T @ K[:t + 1] + lam * np.eye(dk)
        assert np.allclose(kts[t], np.linalg.solve(G, K[t]), atol=1e-10)
        Ct = V[:t + 1].T @ K[:t + 1]
        assert np.allclose(o[t], Ct @ np.linalg.solve(G, Q[t]), atol=1e-9)


def test_external_write_key_from_exact_gram_recovers_least_squares():
    """The main recurrence with k as the read key and an externally given
    write key: feeding it the exact Sherman-Morrison write key (beta = 1,
    no gate) must reproduce the least-squares maps.  Swapping the roles of
    read and write keys, or a transposed update, breaks this."""
    rng = np.random.default_rng(7)
    T, dk, dv, lam = 16, 5, 4, 0.5
    K = rng.standard_normal((T, dk))
    V = rng.standard_normal((T, dv))
    Q = rng.standard_normal((T, dk))
    _, kts, _, _ = recurrent.exact_gram_pdn(K, V, Q, lam)
    o, S_T, S_all = recurrent.delta_rule(
        Q[None], K[None], kts[None], V[None], np.ones((1, T)),
        return_states=True)
    L = lsq.ridge_maps(K, V, lam)
    assert np.abs(S_all[0] - L).max() < 1e-10
    assert np.abs(o[0] - np.einsum("tvk,tk->tv", L, Q)).max() < 1e-10


# ---------------------------------------------------------------- App. B
def _golden(name):
    out = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, *vals = line.split()
        out[key] = np.array([float(x) for x in vals])
    return out


def test_worked_example_apdn_vs_apla():
    """App. B: lambda = 1, k_1 = v_1 = [1,1] gives S^APDN_1 = 1/3 11^T and
    S^APLA_1 = 1/2 11^T (values printed in the paper)."""
    gd = _golden("worked_example.txt")
    lam = float(gd["lambda"][0])
    k1, v1 = gd["k1"][None], gd["v1"][None]
    q = np.array([[1.0, 0.0]])
    S_pdn, kt, _ = recurrent.diag_sm_pdn(k1, v1, q, lam)
    M_pla, _ = recurrent.atq_pla(k1, v1, q, lam)
    assert np.allclose(kt[0], gd["kt1"], atol=1e-15)
    assert np.allclose(S_pdn[0].ravel(), gd["S_APDN_1"], atol=1e-15)
    assert np.allclose(M_pla[0].ravel(), gd["S_APLA_1"], atol=1e-15)


def test_diag_sm_write_key_bounded():
    """App. B "Stability of write-key formulation": with the normalised
    (Sherman-Morrison) diagonal write key, 0 <= k^T kt <= 1 for any key."""
    rng = np.random.default_rng(3)
    K = rng.standard_normal((200, 6)) * np.exp(rng.standard_normal((200, 1)))
    _, kts, _ = recurrent.diag_sm_pdn(K, rng.standard_normal((200, 2)),
                                      K, lam=0.3)
    kk = np.einsum("td,td->t", K, kts)
    assert kk.min() >= 0.0 and kk.max() <= 1.0


def test_general_modes_on_worked_example():
    """The end-to-end oracle's Sherman-Morrison (diag_sm) and apply-to-query
    (atq) modes reproduce the paper's printed values of App. B's worked
    example (lambda = 1, k_1 = v_1 = [1, 1], beta = beta^P = 1, no decay):
    kt_1 = 1/3 1, S^APDN_1 = 1/3 11^T and the read-out map 1/2 11^T."""
    gd = _golden("worked_example.txt")
    lam = float(gd["lambda"][0])
    k = gd["k1"][None, None]
    v = gd["v1"][None, None]
    one = np.ones((1, 1))
    for qv in ([1.0, 0.0], [0.0, 1.0]):
        q = np.array(qv)[None, None]
        r = recurrent.pdn_forward(q, k, v, one, precond="diag_sm", beta_p=one,
                                  ridge=lam)
        assert np.allclose(r["kt"][0, 0], gd["kt1"], atol=1e-15)
        assert np.allclose(r["S_T"][0].ravel(), gd["S_APDN_1"], atol=1e-15)
        ra = recurrent.pdn_forward(q, k, v, one, precond="atq", beta_p=one,
                                   ridge=lam)
        # o_1 = M_1 q with M_1 = S^APLA_1
        M = gd["S_APLA_1"].reshape(2, 2)
        assert np.allclose(ra["o"][0, 0], M @ np.array(qv), atol=1e-15)


def _mode_inputs(rng, T, dk, dv, N=2):
    k = rng.standard_normal((N, T, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    q = rng.standard_normal((N, T, dk))
    v = rng.standard_normal((N, T, dv))
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((N, T))))
    return q, k, v, beta


def test_diag_sm_general_matches_single_head_form():
    """With beta, beta^P, g^P and A0 all drawn at random (no gate), the
    end-to-end diag_sm mode equals the single-head Sherman-Morrison
    recurrence pinned above, head by head."""
    rng = np.random.default_rng(21)
    q, k, v, beta = _mode_inputs(rng, 40, 5, 3)
    bp = rng.uniform(0.1, 2.0, (2, 40))
    gp = -0.2 * rng.uniform(size=(2, 40))
    A0 = rng.uniform(0.0, 1.0, (2, 5))
    r = recurrent.pdn_forward(q, k, v, beta, precond="diag_sm", beta_p=bp,
                              g_p=gp, A0=A0, ridge=0.3)
    for n in range(2):
        S_all, kts, o = recurrent.diag_sm_pdn(k[n], v[n], q[n], 0.3,
                                              beta=beta[n], beta_p=bp[n],
                                              g_p=gp[n], A0=A0[n])
        assert np.allclose(r["kt"][n], kts, rtol=1e-13, atol=1e-15)
        assert np.allclose(r["o"][n], o, rtol=1e-12, atol=1e-13)
        assert np.allclose(r["S_T"][n], S_all[-1], rtol=1e-12, atol=1e-13)
    kk = np.einsum("ntd,ntd->nt", k, r["kt"])
    assert kk.min() >= 0.0 and kk.max() <= 1.0      # App. B stability bound


def test_atq_general_matches_pla_form():
    """With a scalar decay (P-Mamba-2) and beta^P = 1, g^P absent, the
    end-to-end atq mode equals the single-head preconditioned linear
    attention read-out pinned above."""
    rng = np.random.default_rng(22)
    q, k, v, beta = _mode_inputs(rng, 40, 5, 3)
    g = -0.1 * np.log1p(np.exp(rng.standard_normal((2, 40))))
    r = recurrent.pdn_forward(q, k, v, beta, g=g, gate="scalar",
                              precond="atq", beta_p=np.ones((2, 40)),
                              ridge=0.7, scale=0.5)
    for n in range(2):
        _, o = recurrent.atq_pla(k[n], v[n], q[n], 0.7, beta=beta[n], g=g[n])
        assert np.allclose(r["o"][n], 0.5 * o, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("precond", ["diag_sm", "atq"])
def test_channel_gate_with_equal_channels_is_scalar_gate(precond):
    """A per-channel decay whose channels all carry the same value is the
    scalar decay: both general modes agree exactly under the two gates."""
    rng = np.random.default_rng(23)
    q, k, v, beta = _mode_inputs(rng, 30, 4, 3)
    g = -0.2 * rng.uniform(size=(2, 30))
    gc = np.repeat(g[:, :, None], 4, axis=2)
    kw = dict(precond=precond, beta_p=rng.uniform(0.1, 1.0, (2, 30)),
              g_p=-0.1 * rng.uniform(size=(2, 30)), ridge=0.4)
    a = recurrent.pdn_forward(q, k, v, beta, g=g, gate="scalar", **kw)
    b = recurrent.pdn_forward(q, k, v, beta, g=gc, gate="channel", **kw)
    assert np.allclose(a["o"], b["o"], rtol=1e-13, atol=1e-14)
    assert np.allclose(a["S_T"], b["S_T"], rtol=1e-13, atol=1e-14)


def test_knorm_factors_reduce_at_x_1():
    """x = 1 makes B = 1, so with unit keys m_t = 1 and the normalisation
    ablation's factors become constants: 1/m = 1 (the identity write key),
    1/(1+m) = 1/2 and beta/(alpha + beta m) = beta/(alpha + beta), each an
    external write key written in closed form."""
    rng = np.random.default_rng(24)
    q, k, v, beta = _mode_inputs(rng, 30, 4, 3)
    g = -0.3 * rng.uniform(size=(2, 30))
    kw = dict(g=g, gate="scalar", beta_p=rng.uniform(0.1, 1.0, (2, 30)),
              g_p=-0.1 * rng.uniform(size=(2, 30)), x=1.0)
    ident = recurrent.pdn_forward(q, k, v, beta, precond="identity", g=g,
                                  gate="scalar")
    r = recurrent.pdn_forward(q, k, v, beta, knorm="m", **kw)
    assert np.allclose(r["o"], ident["o"], rtol=1e-12, atol=1e-13)
    half = recurrent.pdn_forward(q, k, v, beta, precond="external",
                                 kt_ext=0.5 * k, g=g, gate="scalar")
    r = recurrent.pdn_forward(q, k, v, beta, knorm="1pm", **kw)
    assert np.allclose(r["o"], half["o"], rtol=1e-12, atol=1e-13)
    fac = (beta / (np.exp(g) + beta))[..., None]
    ext = recurrent.pdn_forward(q, k, v, beta, precond="external",
                                kt_ext=fac * k, g=g, gate="scalar")
    r = recurrent.pdn_forward(q, k, v, beta, knorm="beta", **kw)
    assert np.allclose(r["o"], ext["o"], rtol=1e-12, atol=1e-13)


def test_knorm_invariants():
    """With the squash gain in force (x = 1.5, keys of varied norm): the 1/m
    factor makes k^T kt = 1 exactly and the 1/(1+m) factor keeps it in
    [0, 1)."""
    rng = np.random.default_rng(25)
    q, k, v, beta = _mode_inputs(rng, 50, 6, 2)
    k = k * np.exp(rng.standard_normal((2, 50, 1)))
    kw = dict(beta_p=rng.uniform(0.01, 2.0, (2, 50)), x=1.5)
    r = recurrent.pdn_forward(q, k, v, beta, knorm="m", **kw)
    assert np.allclose(np.sum(k * r["kt"], axis=-1), 1.0, rtol=1e-13)
    r = recurrent.pdn_forward(q, k, v, beta, knorm="1pm", **kw)
    kk = np.sum(k * r["kt"], axis=-1)
    assert kk.min() >= 0.0 and kk.max() < 1.0


@pytest.mark.parametrize("gate", ["none", "scalar"])
def test_knorm_beta_factor_is_decayed_sherman_morrison(gate):
    """The beta/(alpha + beta m) factor is the decayed Sherman-Morrison
    normaliser (App. B, Sherman-Morrison update of the inverse Gram, with a
    decay alpha and gain beta): for G_t = alpha G_{t-1} + beta k k^T and
    P = G_{t-1}^{-1},
        beta G_t^{-1} k = beta / (alpha + beta k^T P k) * P k.
    The oracle's factor, handed the write key P k for a random dense SPD
    G_{t-1} (not diagonal), must reproduce the dense inverse on the left."""
    rng = np.random.default_rng(26)
    dk, T = 6, 8
    k = rng.standard_normal((1, T, dk))
    beta = rng.uniform(0.1, 2.0, (1, T))
    g = None if gate == "none" else -rng.uniform(0.0, 1.0, (1, T))
    kt = np.empty_like(k)
    ref = np.empty_like(k)
    for t in range(T):
        Z = rng.standard_normal((dk, dk))
        G = Z @ Z.T + 0.5 * np.eye(dk)
        kt[0, t] = np.linalg.inv(G) @ k[0, t]
        al = 1.0 if g is None else np.exp(g[0, t])
        Gt = al * G + beta[0, t] * np.outer(k[0, t], k[0, t])
        ref[0, t] = beta[0, t] * np.linalg.inv(Gt) @ k[0, t]
    fac = recurrent.knorm_factor(k, kt, beta, g, gate, "beta")
    assert np.allclose(fac * kt, ref, rtol=1e-10, atol=1e-12)


def test_knorm_1pm_factor_is_sherman_morrison():
    """The 1/(1 + m) factor is the undecayed, unit-gain Sherman-Morrison
    normaliser (App. B): with P = G^{-1}, (G + k k^T)^{-1} k =
    P k / (1 + k^T P k), checked against a dense inverse."""
    rng = np.random.default_rng(27)
    dk, T = 5, 6
    k = rng.standard_normal((1, T, dk))
    kt = np.empty_like(k)
    ref = np.empty_like(k)
    for t in range(T):
        Z = rng.standard_normal((dk, dk))
        G = Z @ Z.T + 0.3 * np.eye(dk)
        kt[0, t] = np.linalg.solve(G, k[0, t])
        ref[0, t] = np.linalg.solve(G + np.outer(k[0, t], k[0, t]), k[0, t])
    fac = recurrent.knorm_factor(k, kt, np.ones((1, T)), None, "none", "1pm")
    assert np.allclose(fac * kt, ref, rtol=1e-10, atol=1e-12)


# ------------------------------------- App. D linear attention (ATQ family)
def _la_decays(rng, gate, N, T, dk, strength=0.3):
    if gate == "none":
        return None, np.ones((N, T, dk))
    if gate == "scalar":
        g = -strength * rng.uniform(size=(N, T))
        return g, np.repeat(np.exp(g)[..., None], dk, axis=2)
    g = -strength * rng.uniform(size=(N, T, dk))
    return g, np.exp(g)


@pytest.mark.parametrize("gate", ["none", "scalar", "channel"])
def test_decayed_linear_attention_unrolled_closed_form(gate):
    """S_t = alpha_t S_{t-1} + beta_t v_t k_t^T unrolls to
        S_t = S0 Diag(D_{0,t}) + sum_{j<=t} beta_j v_j (k_j * D_{j,t})^T,
    D_{j,t} = prod_{j<m<=t} alpha_m (the new term is not decayed by its own
    alpha_j), and o_t = scale S_t q_t: the quadratic (attention) form of
    Mamba-2 / GLA.  Brute force over (t, j) with explicit products, against
    the oracle's token recurrence, on tiny inputs."""
    rng = np.random.default_rng(61)
    N, T, dk, dv = 1, 12, 4, 3
    q = rng.standard_normal((N, T, dk))
    k = rng.standard_normal((N, T, dk))
    v = rng.standard_normal((N, T, dv))
    beta = rng.uniform(0.0, 2.0, (N, T))
    S0 = rng.standard_normal((N, dv, dk))
    g, alpha = _la_decays(rng, gate, N, T, dk)
    o, S_T = recurrent.linear_attention(q, k, v, beta, g, gate, S0, scale=0.7)

    def D(j, t):          # prod of alpha over 1-based tokens j+1..t
        return np.prod(alpha[0, j:t], axis=0)

    for t in range(1, T + 1):
        S = S0[0] * D(0, t)[None, :]
        for j in range(1, t + 1):
            S = S + beta[0, j - 1] * np.outer(v[0, j - 1], k[0, j - 1] * D(j, t))
        assert np.allclose(o[0, t - 1], 0.7 * S @ q[0, t - 1], rtol=1e-12,
                           atol=1e-12)
    assert np.allclose(S_T[0], S, rtol=1e-12, atol=1e-12)


def test_linear_attention_is_causal_masked_product():
    """No decay, unit gain, zero initial state: the linear-attention outputs
    are the causal masked product O = (tril(Q K^T)) V (the textbook identity
    behind App. D's PLA form with the whole sequence as one chunk), with
    tril from the library."""
    rng = np.random.default_rng(62)
    q = rng.standard_normal((2, 20, 5))
    k = rng.standard_normal((2, 20, 5))
    v = rng.standard_normal((2, 20, 3))
    o, _ = recurrent.linear_attention(q, k, v, np.ones((2, 20)))
    ref = np.tril(q @ np.swapaxes(k, 1, 2)) @ v
    assert np.allclose(o, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("gate", ["none", "scalar", "channel"])
@pytest.mark.parametrize("C", [1, 2, 4, 8, 16, 32, 64])
def test_la_chunkwise_equals_recurrent(gate, C):
    """App. D's PLA / P-Mamba-2 / PGLA chunkwise forms equal the token
    recurrence of (decayed) linear attention, with a gain, a ragged last
    chunk and S0 != 0."""
    rng = np.random.default_rng(63 + C)
    N, T, dk, dv = 2, 100, 8, 6
    q = rng.standard_normal((N, T, dk))
    k = _unit(rng.standard_normal((N, T, dk)))
    v = rng.standard_normal((N, T, dv))
    beta = _sig(rng.standard_normal((N, T)))
    S0 = 0.1 * rng.standard_normal((N, dv, dk))
    g, _ = _la_decays(rng, gate, N, T, dk, strength=0.2)
    o, S_T = recurrent.linear_attention(q, k, v, beta, g, gate, S0, scale=0.8)
    o2, S2 = chunkwise.la_chunk_forward(q, k, v, beta, g, gate, S0, C, 0.8)
    assert np.abs(o - o2).max() <= 1e-12 * np.abs(o).max()
    assert np.abs(S_T - S2).max() <= 1e-12 * np.abs(S_T).max()


@pytest.mark.parametrize("gate", ["none", "scalar", "channel"])
def test_atq_end_to_end_equals_chunkwise_forms(gate):
    """The apply-to-query mode over many tokens with decays, gains, A0 and
    S0: the oracle's end-to-end result equals App. D's composition of the
    chunkwise Gram recurrence (Eq. precond_from_boundary) with the
    chunkwise P-Mamba-2 / PGLA forms applied to q / (A_t + ridge)."""
    rng = np.random.default_rng(64)
    N, T, dk, dv = 2, 90, 6, 5
    q = _unit(rng.standard_normal((N, T, dk)))
    k = _unit(rng.standard_normal((N, T, dk)))
    v = rng.standard_normal((N, T, dv))
    beta = _sig(rng.standard_normal((N, T)))
    g, _ = _la_decays(rng, gate, N, T, dk, strength=0.2)
    bp = rng.uniform(0.1, 2.0, (N, T))
    gp = -0.1 * rng.uniform(size=(N, T))
    A0 = rng.uniform(0.0, 1.0, (N, dk))
    S0 = 0.1 * rng.standard_normal((N, dv, dk))
    r = recurrent.pdn_forward(q, k, v, beta, g=g, gate=gate, precond="atq",
                              beta_p=bp, g_p=gp, A0=A0, S0=S0, ridge=0.4,
                              scale=1.1)
    A_all, A_bound = chunkwise.gram_chunkwise(k, bp, gp, 16, A0)
    o2, S2 = chunkwise.la_chunk_forward(q / (A_all + 0.4), k, v, beta, g, gate,
                                        S0, 16, 1.1)
    assert np.abs(r["o"] - o2).max() <= 1e-12 * np.abs(r["o"]).max()
    assert np.abs(r["S_T"] - S2).max() <= 1e-12 * np.abs(r["S_T"]).max()
    assert np.allclose(r["A_T"], A_bound[:, -1], rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- Sec. 3.5
def test_squash_range_monotone_and_fixed_points():
    """Eq. precond_end2end: B in [1/x, x], decreasing in A, B = 1 where
    log A = mu, and x = 1 gives B = 1 exactly."""
    A = np.concatenate([[0.0], np.logspace(-30, 30, 2001)])
    for x in (1.25, 1.5, 2.0):
        for mu in (0.2, 1.0, 3.0):
            B = recurrent.squash(A, mu, x)
            assert B.max() <= x * (1 + 1e-15) and B.min() >= (1 / x) * (1 - 1e-15)
            assert np.all(np.diff(B) <= 0)
            assert B[0] == pytest.approx(x)          # A = 0 limit
            assert recurrent.squash(np.exp(mu), mu, x) == pytest.approx(1.0)
    assert np.all(recurrent.squash(A, 1.0, 1.0) == 1.0)


def test_squash_worked_values():
    """s = r/(1+|r|) at r = +-1 is +-1/2, so B = x^{-1/2} / x^{1/2}."""
    x = 1.5
    assert recurrent.squash(np.exp(2.0), 1.0, x) == pytest.approx(x ** -0.5)
    assert recurrent.squash(np.exp(0.0), 1.0, x) == pytest.approx(x ** 0.5)


def test_preconditioner_scan_closed_forms():
    """Eq. diag_gram: with alpha^P = 1 the state is the running sum of
    beta^P k*k (numpy cumsum); with a constant decay it is the geometric
    sum."""
    rng = np.random.default_rng(11)
    N, T, dk = 2, 40, 7
    k = rng.standard_normal((N, T, dk))
    bp = rng.uniform(0.1, 2.0, (N, T))
    A0 = rng.uniform(0, 1, (N, dk))
    _, A_all, A_T = recurrent.preconditioner_scan(k, bp, None, np.ones(N),
                                                  1.5, A0)
    ref = A0[:, None] + np.cumsum(bp[..., None] * k ** 2, axis=1)
    assert np.allclose(A_all, ref, rtol=1e-13)
    c = -0.2
    _, A_all, _ = recurrent.preconditioner_scan(k, bp, np.full((N, T), c),
                                                np.ones(N), 1.5, A0)
    t = np.arange(T)
    w = np.exp(c * (t[:, None] - t[None, :])) * (t[:, None] >= t[None, :])
    ref = np.exp(c * (t + 1))[None, :, None] * A0[:, None] + np.einsum(
        "ts,nsd->ntd", w, bp[..., None] * k ** 2)
    assert np.allclose(A_all, ref, rtol=1e-12)


def test_kt_k_bounded_for_unit_keys():
    """App. E Lemma (unit-disk eigenvalues): for ||k|| = 1 and B in
    [1/x, x], k^T kt lies in [1/x, x]."""
    rng = np.random.default_rng(5)
    N, T, dk = 4, 300, 16
    k = _unit(rng.standard_normal((N, T, dk)) * np.exp(
        2 * rng.standard_normal((1, 1, dk))))
    bp = 10.0 ** rng.uniform(-4, 4, (N, T))
    kt, _, _ = recurrent.preconditioner_scan(k, bp, None, np.ones(N), 1.5)
    kk = np.einsum("ntd,ntd->nt", k, kt)
    assert kk.min() >= 1 / 1.5 - 1e-12 and kk.max() <= 1.5 + 1e-12
    assert kk.min() < 0.8 and kk.max() > 1.3     # both sides of 1 reached


@pytest.mark.parametrize("gate", ["none", "scalar", "channel"])
def test_x_equal_one_reduces_to_identity(gate):
    """x = 1 makes B = 1, so PDN/PGDN/PKDA become DN/GDN/KDA exactly."""
    rng = np.random.default_rng(13)
    q, k, v, beta, g, bp, gp, mu = _rand_problem(rng, 2, 30, 6, 5, gate)
    a = recurrent.pdn_forward(q, k, v, beta, g=g, gate=gate, precond="squash",
                              beta_p=bp, g_p=gp, mu=mu, x=1.0)
    b = recurrent.pdn_forward(q, k, v, beta, g=g, gate=gate,
                              precond="identity")
    assert np.array_equal(a["o"], b["o"]) and np.array_equal(a["S_T"], b["S_T"])


# ------------------------------------------------- delta-rule closed forms
@pytest.mark.parametrize("gate", ["none", "scalar", "channel"])
def test_orthonormal_keys_closed_form(gate):
    """With orthonormal read/write keys k_t = e_t the read S_{t-1} k_t only
    sees the decayed initial state, and the state has a closed form:
    S_t = S0 D_{0,t} + sum_{i<=t} beta_i (v_i - S0 D_{0,i} e_i) e_i^T D_{i,t}
    with D_{i,t} the decay accumulated over (i, t]."""
    rng = np.random.default_rng(17)
    dk, dv, T = 6, 4, 6
    k = np.eye(dk)[None, :T]
    q = rng.standard_normal((1, T, dk))
    v = rng.standard_normal((1, T, dv))
    beta = rng.uniform(0, 1, (1, T))
    S0 = rng.standard_normal((1, dv, dk))
    if gate == "none":
        alpha = np.ones((T, dk))
        g = None
    elif gate == "scalar":
        g = -rng.uniform(0, 0.5, (1, T))
        alpha = np.repeat(np.exp(g[0])[:, None], dk, 1)
    else:
        g = -rng.uniform(0, 0.5, (1, T, dk))
        alpha = np.exp(g[0])
    o, S_T = recurrent.delta_rule(q, k, k, v, beta, g, gate, S0, scale=0.5)

    def D(i, t):          # decay over tokens i+1..t (1-based), per channel
        return np.prod(alpha[i:t], axis=0)

    for t in range(1, T + 1):
        S = S0[0] * D(0, t)[None]
        for i in range(1, t + 1):
            read = (S0[0] * D(0, i)[None])[:, i - 1]
            S = S + beta[0, i - 1] * np.outer(v[0, i - 1] - read,
                                              np.eye(dk)[i - 1] * D(i, t))
        assert np.allclose(o[0, t - 1], 0.5 * S @ q[0, t - 1], atol=1e-12)
    assert np.allclose(S_T[0], S, atol=1e-12)


def test_unit_key_beta_one_overwrites_association():
    """Delta rule with ||k|| = 1, beta = 1, kt = k: after the write,
    S_t k_t = v_t exactly (the old association along k_t is replaced)."""
    rng = np.random.default_rng(19)
    N, T, dk, dv = 3, 20, 8, 5
    k = _unit(rng.standard_normal((N, T, dk)))
    v = rng.standard_normal((N, T, dv))
    _, _, S_all = recurrent.delta_rule(k, k, k, v, np.ones((N, T)),
                                       return_states=True)
    assert np.abs(np.einsum("ntvk,ntk->ntv", S_all, k) - v).max() < 1e-12


def test_deltanet_error_contracts_in_noiseless_regression():
    """App. B proof of Theorem (DN better approximates least squares than
    LA): with v_t = S* k_t, unit keys and beta in [0,1], ||S* - S_t||_F is
    non-increasing."""
    rng = np.random.default_rng(23)
    N, T, dk, dv = 4, 200, 8, 6
    Sstar = rng.standard_normal((N, dv, dk))
    k = _unit(rng.standard_normal((N, T, dk)))
    v = np.einsum("nvk,ntk->ntv", Sstar, k)
    _, _, S_all = recurrent.delta_rule(k, k, k, v, rng.uniform(0, 1, (N, T)),
                                       return_states=True)
    err = np.linalg.norm(S_all - Sstar[:, None], axis=(2, 3))
    err = np.concatenate([np.linalg.norm(Sstar, axis=(1, 2))[:, None], err], 1)
    assert np.all(np.diff(err, axis=1) <= 1e-12)
    assert err[:, -1].max() < 0.05 * err[:, 0].min()


def test_la_error_closed_form_monte_carlo():
    """App. B Eq. la_err_closed: for unit isotropic keys and queries,
    E||o^LA - o*||^2 = ||S*||^2/d (1 - t/d + t(t-1)/d^2).  Checked by
    Monte Carlo with the oracle's linear-attention read-out (the ATQ mode
    with lam -> 0 is not used; plain C_t q_t)."""
    rng = np.random.default_rng(29)
    d, t, n = 4, 6, 40000
    Sstar = rng.standard_normal((d, d))
    z = rng.standard_normal((n, t, d))
    K = z / np.linalg.norm(z, axis=-1, keepdims=True)
    qz = rng.standard_normal((n, d))
    qv = qz / np.linalg.norm(qz, axis=-1, keepdims=True)
    G = np.einsum("nti,ntj->nij", K, K)
    dev = np.einsum("vk,nkj,nj->nv", Sstar, G - np.eye(d)[None], qv)
    mc = (dev ** 2).sum(1).mean()
    ref = (Sstar ** 2).sum() / d * (1 - t / d + t * (t - 1) / d ** 2)
    assert mc == pytest.approx(ref, rel=0.03)


@pytest.mark.parametrize("gate", ["scalar", "channel"])
def test_transition_eigenvalues(gate):
    """App. E Lemma: the transition alpha (I - beta k kt^T) has eigenvalues
    alpha (multiplicity dk-1) and alpha (1 - beta kt^T k).  The oracle's
    step applied to S_{t-1} = I with v = 0 gives that right factor."""
    rng = np.random.default_rng(31)
    dk = 6
    for _ in range(20):
        k = _unit(rng.standard_normal(dk))
        kt = rng.uniform(1 / 1.5, 1.5, dk) * k
        beta = rng.uniform(0, 1.3)
        if gate == "scalar":
            g = np.array([[-rng.uniform(0, 1)]])
            a = np.exp(g[0, 0])
        else:
            gval = -rng.uniform(0, 1)
            g = np.full((1, 1, dk), gval)
            a = np.exp(gval)
        _, S1 = recurrent.delta_rule(np.zeros((1, 1, dk)), k[None, None],
                                     kt[None, None], np.zeros((1, 1, dk)),
                                     np.array([[beta]]), g, gate,
                                     np.eye(dk)[None])
        ev = np.sort_complex(np.linalg.eigvals(S1[0]))
        ref = np.sort_complex(np.array([a] * (dk - 1) + [a * (1 - beta * kt @ k)],
                                       dtype=complex))
        assert np.allclose(ev, ref, atol=1e-10)
        if beta * 1.5 <= 2:
            assert np.abs(ev).max() <= 1 + 1e-12


@pytest.mark.parametrize("gate", ["none", "scalar", "channel"])
def test_zero_beta_closed_form(gate):
    """beta = 0: nothing is written, the state only decays:
    S_t = S0 Diag(prod_{j<=t} alpha_j) and o_t = scale S_t q_t."""
    rng = np.random.default_rng(37)
    q, k, v, beta, g, bp, gp, mu = _rand_problem(rng, 2, 25, 5, 4, gate)
    S0 = rng.standard_normal((2, 4, 5))
    o, S_T = recurrent.delta_rule(q, k, k, v, np.zeros_like(beta), g, gate,
                                  S0, scale=1.3)
    if gate == "none":
        cum = np.ones((2, 25, 5))
    elif gate == "scalar":
        cum = np.repeat(np.exp(np.cumsum(g, 1))[..., None], 5, 2)
    else:
        cum = np.exp(np.cumsum(g, 1))
    ref_o = 1.3 * np.einsum("nvk,ntk,ntk->ntv", S0, cum, q)
    assert np.allclose(o, ref_o, atol=1e-12)
    assert np.allclose(S_T, S0 * cum[:, -1][:, None, :], atol=1e-12)


# ------------------------------------------------------------ App. D
@pytest.mark.parametrize("gate", ["none", "scalar", "channel"])
@pytest.mark.parametrize("C", [1, 2, 4, 8, 16, 32, 64])
def test_chunkwise_equals_recurrent(gate, C):
    """App. D chunkwise forms (with the gated UT system as read here) equal
    the token recurrence, including a ragged last chunk and S0 != 0."""
    rng = np.random.default_rng(41 + C)
    T = 100
    q, k, v, beta, g, bp, gp, mu = _rand_problem(rng, 2, T, 8, 6, gate)
    S0 = 0.1 * rng.standard_normal((2, 6, 8))
    kt, _, _ = recurrent.preconditioner_scan(k, bp, gp, mu, 1.5)
    o, S_T = recurrent.delta_rule(q, k, kt, v, beta, g, gate, S0, 0.8)
    o2, S2 = chunkwise.chunk_forward(q, k, kt, v, beta, g, gate, S0, C, 0.8)
    assert np.abs(o - o2).max() <= 1e-12 * np.abs(o).max()
    assert np.abs(S_T - S2).max() <= 1e-12 * np.abs(S_T).max()


@pytest.mark.parametrize("C", [1, 7, 16, 64])
def test_preconditioner_chunkwise_equals_scan(C):
    """App. D Eq. precond_from_boundary and the decayed causal mask give the
    same A_t (hence kt) as the token scan; boundary states match."""
    rng = np.random.default_rng(43)
    N, T, dk = 3, 150, 9
    k = rng.standard_normal((N, T, dk))
    bp = rng.uniform(0, 2, (N, T))
    gp = -rng.uniform(0, 0.4, (N, T))
    mu = np.exp(rng.standard_normal(N))
    A0 = rng.uniform(0, 1, (N, dk))
    kt, A_all, A_T = recurrent.preconditioner_scan(k, bp, gp, mu, 1.5, A0)
    kt2, Ab = chunkwise.preconditioner_chunkwise(k, bp, gp, mu, 1.5, C, A0)
    assert np.abs(kt - kt2).max() < 1e-12
    assert np.allclose(Ab[:, -1], A_T, rtol=1e-12)
    assert np.allclose(Ab[:, 1:-1], A_all[:, C - 1:-1:C][:, :Ab.shape[1] - 2],
                       rtol=1e-12)


def test_chunk_intermediates_satisfy_ut_system():
    """W and U solve (I + tril(Diag(beta) K Kt^T, -1)) X = Diag(beta) [K|V]
    (App. D, matrix form of the w/u recurrences), checked by forward
    substitution of the w_r / u_r recurrences (Eq. w_rec_two_key,
    u_rec_two_key) rather than by a solve."""
    rng = np.random.default_rng(47)
    q, k, v, beta, g, bp, gp, mu = _rand_problem(rng, 1, 16, 5, 4, "none")
    kt, _, _ = recurrent.preconditioner_scan(k, bp, gp, mu, 1.5)
    _, _, inter = chunkwise.chunk_forward(q, k, kt, v, beta, C=16, keep=True)
    K, Kt, V, b = k[0], kt[0], v[0], beta[0]
    w = np.zeros_like(K)
    u = np.zeros_like(V)
    for r in range(16):
        w[r] = b[r] * (K[r] - sum(w[t] * (Kt[t] @ K[r]) for t in range(r)))
        u[r] = b[r] * (V[r] - sum(u[t] * (Kt[t] @ K[r]) for t in range(r)))
    assert np.allclose(inter["W"][0], w, atol=1e-12)
    assert np.allclose(inter["U"][0], u, atol=1e-12)


@pytest.mark.parametrize("gate", ["none", "scalar", "channel"])
def test_split_sequence_chaining(gate):
    """Running [0, tau) then [tau, T) while carrying (S, A) equals one
    run over [0, T)."""
    rng = np.random.default_rng(53)
    q, k, v, beta, g, bp, gp, mu = _rand_problem(rng, 2, 90, 6, 4, gate)
    full = recurrent.pdn_forward(q, k, v, beta, g=g, gate=gate, beta_p=bp,
                                 g_p=gp, mu=mu, x=1.5)
    tau = 37
    cut = (lambda a, s: None if a is None else a[:, s])
    first = recurrent.pdn_forward(
        q[:, :tau], k[:, :tau], v[:, :tau], beta[:, :tau],
        g=cut(g, slice(0, tau)), gate=gate, beta_p=bp[:, :tau],
        g_p=gp[:, :tau], mu=mu, x=1.5)
    second = recurrent.pdn_forward(
        q[:, tau:], k[:, tau:], v[:, tau:], beta[:, tau:],
        g=cut(g, slice(tau, None)), gate=gate, beta_p=bp[:, tau:],
        g_p=gp[:, tau:], mu=mu, x=1.5, S0=first["S_T"], A0=first["A_T"])
    assert np.allclose(np.concatenate([first["o"], second["o"]], 1),
                       full["o"], atol=1e-13)
    assert np.allclose(second["S_T"], full["S_T"], atol=1e-13)
    assert np.allclose(second["A_T"], full["A_T"], rtol=1e-13)


# ------------------------------------------------------------ adjoint
@pytest.mark.parametrize("gate,precond", [
    ("none", "squash"), ("scalar", "squash"), ("channel", "squash"),
    ("scalar", "identity"), ("channel", "external")])
def test_adjoint_matches_finite_differences(gate, precond):
    """Every gradient of <dO, o> + <dS_T, S_T> against central finite
    differences of the forward recurrence (float64, h = 1e-6)."""
    rng = np.random.default_rng(59)
    N, T, dk, dv = 2, 6, 4, 3
    q = rng.standard_normal((N, T, dk))
    k = rng.standard_normal((N, T, dk))
    v = rng.standard_normal((N, T, dv))
    do = rng.standard_normal((N, T, dv))
    beta = rng.uniform(0, 1.5, (N, T))
    bp = rng.uniform(0.1, 1, (N, T))
    gp = -rng.uniform(0, 0.3, (N, T))
    mu = np.exp(0.2 * rng.standard_normal(N))
    S0 = rng.standard_normal((N, dv, dk))
    A0 = rng.uniform(0.01, 1, (N, dk))
    dST = rng.standard_normal((N, dv, dk))
    kt_ext = rng.standard_normal((N, T, dk))
    g = None
    if gate == "scalar":
        g = -rng.uniform(0, 0.3, (N, T))
    elif gate == "channel":
        g = -rng.uniform(0, 0.3, (N, T, dk))
    base = dict(q=q, k=k, v=v, beta=beta, g=g, beta_p=bp, g_p=gp, mu=mu,
                S0=S0, A0=A0, kt_ext=kt_ext)

    def loss(a):
        r = recurrent.pdn_forward(a["q"], a["k"], a["v"], a["beta"], g=a["g"],
                                  gate=gate, precond=precond,
                                  beta_p=a["beta_p"], g_p=a["g_p"],
                                  mu=a["mu"], x=1.5, kt_ext=a["kt_ext"],
                                  S0=a["S0"], A0=a["A0"], scale=0.7)
        return (r["o"] * do).sum() + (r["S_T"] * dST).sum()

    gr = adjoint.pdn_backward(q, k, v, beta, do, g=g, gate=gate,
                              precond=precond, beta_p=bp, g_p=gp, mu=mu,
                              x=1.5, kt_ext=kt_ext, S0=S0, A0=A0, scale=0.7,
                              dS_T=dST, ckpt=4)
    names = dict(q="dq", k="dk", v="dv", beta="dbeta", S0="dS0")
    if g is not None:
        names["g"] = "dg"
    if precond == "squash":
        names.update(beta_p="dbeta_p", g_p="dg_p", mu="dmu", A0="dA0")
    if precond == "external":
        names["kt_ext"] = "dkt"
    for nm, gn in names.items():
        arr = base[nm]
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            ap, am = dict(base), dict(base)
            ap[nm] = arr.copy()
            ap[nm][idx] += 1e-6
            am[nm] = arr.copy()
            am[nm][idx] -= 1e-6
            fd[idx] = (loss(ap) - loss(am)) / 2e-6
        err = np.abs(fd - gr[gn]).max() / max(1e-12, np.abs(fd).max())
        assert err < 1e-6, (nm, err)


def test_adjoint_identity_has_no_preconditioner_gradients():
    """x = 1 makes kt = k exactly, so the preconditioner inputs get exactly
    zero gradient (B is constant)."""
    rng = np.random.default_rng(61)
    q, k, v, beta, g, bp, gp, mu = _rand_problem(rng, 2, 12, 4, 3, "scalar")
    do = rng.standard_normal((2, 12, 3))
    r = adjoint.pdn_backward(q, k, v, beta, do, g=g, gate="scalar",
                             precond="squash", beta_p=bp, g_p=gp, mu=mu,
                             x=1.0, ckpt=5)
    assert np.all(r["dbeta_p"] == 0) and np.all(r["dg_p"] == 0)
    assert np.all(r["dmu"] == 0)
    r2 = adjoint.pdn_backward(q, k, v, beta, do, g=g, gate="scalar",
                              precond="identity", ckpt=5)
    assert np.allclose(r["dk"], r2["dk"], atol=1e-14)


def test_zero_key_channel_limit():
    """A key channel that is exactly zero keeps A = 0 there; the write key
    is still finite (B = x limit) and the gradients stay finite."""
    rng = np.random.default_rng(67)
    q, k, v, beta, g, bp, gp, mu = _rand_problem(rng, 1, 10, 4, 3, "none")
    k = k.copy()
    k[:, :, 2] = 0.0
    r = recurrent.pdn_forward(q, k, v, beta, beta_p=bp, g_p=gp, mu=mu, x=1.5)
    assert np.all(np.isfinite(r["o"])) and np.all(r["A_T"][:, 2] == 0)
    gr = adjoint.pdn_backward(q, k, v, beta, rng.standard_normal((1, 10, 3)),
                              beta_p=bp, g_p=gp, mu=mu, x=1.5)
    for key, val in gr.items():
        assert np.all(np.isfinite(val)), key
