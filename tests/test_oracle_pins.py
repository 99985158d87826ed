"""Pins of the fp64 oracle against what the paper and mathematics fix (CPU only).

Each test checks the oracle against something other than itself: closed forms
from the paper's gate analysis, textbook/library routines in special cases,
theorems about the bound, hand-worked values, and an independent brute-force
reading of the decode algorithm on tiny inputs.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
from scipy.optimize import minimize_scalar
from scipy.special import expit, lambertw

import brute
import oracle
from synth import as_numpy, config1, make_workload

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "gate_regimes.json")))


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    return as_numpy(torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16))


def _f64(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# --------------------------------------------------------------------- gate

@pytest.mark.parametrize("beta,tau", [(1.0, 0.5), (4.0, 2.0), (5.0, 2.81), (2.0, -3.0), (4.0, 0.0),
                                      (4.0, -0.5)])
def test_gate_derivative_at_tau_matches_closed_form(beta, tau):
    h = 1e-6
    num = (oracle.gate(tau + h, tau, beta) - oracle.gate(tau - h, tau, beta)) / (2 * h)
    expected = eval(GOLD["derivative_at_tau"], {}, {"beta": beta, "tau": tau})
    assert abs(num - expected) < 1e-6


@pytest.mark.parametrize("beta,tau", [(4.0, 2.0), (5.0, 2.81), (1.0, 0.3), (5.0, 0.01), (2.0, 1.0)])
def test_gate_minimiser_is_lambert_w_closed_form(beta, tau):
    w = float(lambertw(math.exp(-1.0 - beta * tau)).real)
    s_star = -(1.0 + w) / beta
    res = minimize_scalar(lambda S: oracle.gate(S, tau, beta),
                          bracket=(-3.0 / beta, -1.1 / beta, 0.0), tol=1e-12)
    assert abs(res.x - s_star) < 1e-5
    assert abs(oracle.gate(s_star, tau, beta) - (-w / beta)) < 1e-12
    # footnote bounds on the minimiser for tau > 0
    assert GOLD["sstar_lower_times_beta"] / beta < s_star < GOLD["sstar_upper_times_beta"] / beta


def test_lambert_constant_of_the_footnote():
    w = float(lambertw(math.exp(-1.0)).real)
    assert round(w, GOLD["lambertw0_at_inv_e_decimals"]) == GOLD["lambertw0_at_inv_e"]


def test_gate_shape_limits_and_regimes():
    beta, tau = GOLD["final_beta"], GOLD["trained_median_tau"]
    # far below threshold the gated score contracts to zero (weight exp(0) = 1)
    assert abs(oracle.gate(-40.0, tau, beta)) < 1e-60
    # far above threshold the gate is the identity
    assert abs(oracle.gate(tau + 20.0, tau, beta) - (tau + 20.0)) < 1e-30
    # tau = -inf means no gating at all
    for S in (-3.0, 0.0, 2.5):
        assert oracle.gate(S, -math.inf, beta) == S
    # regime 1 (tau far below -2/beta, e.g. the start-dense bias): essentially dense on the support
    tau1 = GOLD["start_dense_bias"]
    assert tau1 < GOLD["regime1_tau_upper_times_beta"] / beta
    assert max(abs(oracle.gate(S, tau1, beta) - S) for S in np.linspace(-3, 3, 61)) < 1e-8
    # monotone increasing on [S*, inf)
    w = float(lambertw(math.exp(-1.0 - beta * tau)).real)
    grid = np.linspace(-(1 + w) / beta, 10.0, 500)
    vals = oracle.gate_vec(grid, tau, beta)
    assert np.all(np.diff(vals) > 0)


def test_gate_is_logistic_times_score():
    # scipy's logistic function is an independent evaluation of sigma
    for S in (-5.0, -0.3, 0.0, 1.7, 4.0):
        for tau, beta in ((2.0, 4.0), (-1.0, 1.0), (2.81, 5.0)):
            assert abs(oracle.gate(S, tau, beta) - S * expit(beta * (S - tau))) < 1e-14


# ---------------------------------------------------------------- summaries

@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("b", [4, 16, 64])
def test_summaries_match_numpy(dt, b):
    rng = np.random.default_rng(7)
    K = rng.standard_normal((1000, 64)).astype(np.float32) * 1.5 + 0.7
    Kin = K if dt == "f32" else _bf16_bits(K)
    Kd = _f64(Kin)
    mu, sg, M = oracle.summaries(Kin, b)
    N = 1000 // b
    assert mu.shape == (N, 64) and M.shape == (N,)
    blocks = Kd[:N * b].reshape(N, b, 64)
    np.testing.assert_allclose(mu, blocks.mean(axis=1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(sg, blocks.std(axis=1, ddof=0), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(M, np.linalg.norm(blocks, axis=2).max(axis=1), rtol=1e-12)


def test_summaries_population_variance_hand_example():
    # two-token block {x, y}: population std is |x - y| / 2 (not / sqrt(2))
    K = np.array([[3.0, -1.0, 0.0], [1.0, -1.0, 4.0]], np.float32)
    mu, sg, M = oracle.summaries(K, 2)
    np.testing.assert_allclose(mu[0], [2.0, -1.0, 2.0])
    np.testing.assert_allclose(sg[0], [1.0, 0.0, 2.0])
    assert M[0] == pytest.approx(math.sqrt(18.0))   # rows have norms sqrt(10), sqrt(18)


def test_envelope_dominates_flat_sigma_and_hand_case():
    rng = np.random.default_rng(3)
    K = rng.standard_normal((640, 32)).astype(np.float32)
    K[100:104] += 9.0                          # a localised 4-token spike
    mu, sg, _ = oracle.summaries(K, 64)
    env = oracle.envelope(K, 64, 4, mu)
    assert np.all(env >= sg - 1e-12)
    assert np.all(env[1] > 2.0 * sg[1].mean())  # the spike's block is inflated
    # constant sub-blocks: envelope_i = max_m |c_m - mu_i|
    c = np.array([1.0, 2.0, 4.0, 9.0], np.float32)
    Kc = np.repeat(c, 4)[:, None].repeat(3, axis=1).astype(np.float32)
    m2, s2, _ = oracle.summaries(Kc, 16)
    e2 = oracle.envelope(Kc, 16, 4, m2)
    np.testing.assert_allclose(e2[0], np.abs(c - c.mean()).max() * np.ones(3), rtol=1e-12)


# -------------------------------------------------------------------- bound

def test_bound_hand_worked_example():
    # d = 4, q = e1, block {2 e1, 0}: mu = e1, sigma = e1, M = 2
    q = np.array([1.0, 0.0, 0.0, 0.0])
    mu = np.array([1.0, 0.0, 0.0, 0.0]); sg = np.array([1.0, 0.0, 0.0, 0.0])
    assert oracle.bound(q, mu, sg, 2.0, 0.5) == pytest.approx(0.75)   # min(1.5, 2) / 2
    assert oracle.bound(q, mu, sg, 2.0, 2.0) == pytest.approx(1.0)    # min(3, 2) / 2
    q2 = np.array([0.0, 2.0, 0.0, 0.0])                             # orthogonal query
    assert oracle.bound(q2, mu, sg, 2.0, 3.0) == pytest.approx(0.0)


def _random_blocks(seed, nblk, b, d, dt="f32"):
    rng = np.random.default_rng(seed)
    K = rng.standard_normal((nblk * b, d)).astype(np.float32)
    # heavy-tailed coordinates and a few planted, query-aligned blocks
    K[:, 3] *= 4.0
    q = rng.standard_normal(d)
    for j in rng.choice(nblk, nblk // 10, replace=False):
        K[j * b:(j + 1) * b] += (3.0 * math.sqrt(d) * q / np.linalg.norm(q)).astype(np.float32)
    Kin = K if dt == "f32" else _bf16_bits(K)
    return q, Kin


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_spherical_ceiling_is_a_true_upper_bound(dt):
    # with z huge the bound is the Cauchy-Schwarz term |q| M / sqrt(d) >= max_k q.k / sqrt(d)
    b, d = 16, 32
    q, K = _random_blocks(11, 400, b, d, dt)
    mu, sg, M = oracle.summaries(K, b)
    Kd = _f64(K).reshape(400, b, d)
    true_max = (Kd @ q).max(axis=1) / math.sqrt(d)
    for j in range(400):
        bd = oracle.bound(q, mu[j], sg[j], M[j], 1e12)
        assert bd == pytest.approx(np.linalg.norm(q) * M[j] / math.sqrt(d), rel=1e-12)
        assert bd >= true_max[j] - 1e-12


@pytest.mark.parametrize("b,d", [(4, 8), (16, 32), (64, 64)])
def test_dual_bound_is_certified_at_samuelson_diagonal_z(b, d):
    # qT Sigma q <= d sum q_i^2 sigma_i^2 (Cauchy-Schwarz) and Samuelson's
    # inequality (max deviation <= sqrt(b-1) std) => bound >= block max at z = sqrt((b-1) d)
    nblk = 300
    q, K = _random_blocks(5 + b, nblk, b, d)
    mu, sg, M = oracle.summaries(K, b)
    Kd = _f64(K).reshape(nblk, b, d)
    true_max = (Kd @ q).max(axis=1) / math.sqrt(d)
    z = math.sqrt((b - 1) * d)
    for j in range(nblk):
        assert oracle.bound(q, mu[j], sg[j], M[j], z) >= true_max[j] - 1e-12


def test_cantelli_finite_population_count():
    # with the full covariance, at most floor(b / (1 + z^2)) keys exceed mu.q + z sqrt(qT Sigma q)
    b, d = 64, 16
    q, K = _random_blocks(21, 200, b, d)
    mu, sg, M = oracle.summaries(K, b)
    Kd = _f64(K).reshape(200, b, d)
    for z in (0.5, 1.0, 2.0, 3.0):
        cap = math.floor(b / (1 + z * z))
        for j in range(200):
            X = Kd[j] @ q
            cov = np.cov(Kd[j].T, bias=True)
            thr = q @ mu[j] + z * math.sqrt(q @ cov @ q)
            assert int((X >= thr + 1e-9).sum()) <= cap


# ---------------------------------------------------------------- predictor

def test_predictor_special_cases():
    rng = np.random.default_rng(2)
    B, Hq, d = 3, 4, 8
    q = rng.standard_normal((B, Hq, d)).astype(np.float32)
    bias = rng.standard_normal(Hq).astype(np.float32)
    np.testing.assert_array_equal(oracle.predict(q, None, bias), np.tile(bias.astype(np.float64), (B, 1)))
    # one-hot column picks one coordinate of the concatenated query: head 2, dim 5 -> head 1
    W = np.zeros((Hq * d, Hq), np.float32)
    W[2 * d + 5, 1] = 1.0
    W[0 * d + 0, 3] = -2.0
    tau = oracle.predict(q, W, bias)
    np.testing.assert_allclose(tau[:, 1], q[:, 2, 5].astype(np.float64) + bias[1], rtol=0, atol=1e-12)
    np.testing.assert_allclose(tau[:, 3], -2.0 * q[:, 0, 0].astype(np.float64) + bias[3], atol=1e-12)
    np.testing.assert_allclose(tau[:, 0], bias[0], atol=0)
    # linear in W
    W1 = rng.standard_normal((Hq * d, Hq)).astype(np.float32)
    W2 = rng.standard_normal((Hq * d, Hq)).astype(np.float32)
    lhs = oracle.predict(q, W1 + W2, None)
    rhs = oracle.predict(q, W1, None) + oracle.predict(q, W2, None)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-5, atol=1e-5)


def test_start_dense_initialisation_keeps_every_block():
    wl = make_workload(B=1, Hq=4, Hkv=2, d=32, block=16, seq_lens=[512], dtype=torch.float32,
                       predictor=False, tau_const=GOLD["start_dense_bias"], seed=9)
    q, k, v = as_numpy(wl.q), as_numpy(wl.k), as_numpy(wl.v)
    tau = oracle.predict(q, np.zeros((4 * 32, 4), np.float32), as_numpy(wl.bias))
    r = oracle.decode(q, k, v, wl.seq_lens, tau, block_size=16, rescue_window=128)
    assert r.sel.all()
    assert np.all(r.counts == 512)


# ---------------------------------------------------------------- selection

def test_selection_threshold_pins_and_rescue():
    bounds = np.array([0.1, 0.9, 0.9, 0.3, 5.0, 0.2])
    sel, r = oracle.select(bounds, 1.0, c=4)           # nothing >= 1 inside window [0, 4)
    assert r == 1                                      # first of the tied maxima
    np.testing.assert_array_equal(sel, [0, 1, 0, 0, 1, 0])
    sel, r = oracle.select(bounds, 0.5, c=4)           # window already has selections
    assert r == -1
    np.testing.assert_array_equal(sel, [0, 1, 1, 0, 1, 0])
    sel, r = oracle.select(bounds, 10.0, c=2, lwb=1)   # pin outside window, rescue in [0, 2)
    assert r == 1
    np.testing.assert_array_equal(sel, [0, 1, 0, 0, 0, 1])
    sel, r = oracle.select(bounds, 10.0, c=6, lwb=1)   # pinned block inside window: no rescue
    assert r == -1
    np.testing.assert_array_equal(sel, [0, 0, 0, 0, 0, 1])
    sel, r = oracle.select(bounds, 10.0, c=0)          # rescue disabled
    assert r == -1 and sel.sum() == 0
    sel, r = oracle.select(bounds, 0.9, c=4)           # bound == tau survives (>=)
    np.testing.assert_array_equal(sel, [0, 1, 1, 0, 1, 0])
    sel, r = oracle.select(np.array([np.nan, 0.2, np.nan]), 1.0, c=3)
    assert r == 1 and sel.tolist() == [0, 1, 0]
    sel, r = oracle.select(bounds, 10.0, c=6, screen_all=True)
    assert r == -1 and sel.all()


# ---------------------------------------------------------------- attention

def _sdpa(q, K, V, bias=None):
    qt = torch.from_numpy(q)[None, None, None, :]
    kt = torch.from_numpy(K)[None, None]
    vt = torch.from_numpy(V)[None, None]
    m = None if bias is None else torch.from_numpy(bias)[None, None, None, :]
    return torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=m)[0, 0, 0].numpy()


@pytest.mark.parametrize("T", [1, 63, 64, 200, 1000])
def test_tau_minus_inf_is_textbook_softmax_attention(T):
    wl = make_workload(B=2, Hq=4, Hkv=2, d=32, block=16, seq_lens=[T, max(1, T // 2)],
                       T_cap=T, dtype=torch.float32, predictor=False, tau_const=-math.inf,
                       planted={"frac": 0.1}, seed=T)
    q, k, v = as_numpy(wl.q), as_numpy(wl.k), as_numpy(wl.v)
    tau = np.full((2, 4), -np.inf)
    r = oracle.decode(q, k, v, wl.seq_lens, tau, block_size=16, rescue_window=128)
    for bb in range(2):
        Tb = wl.seq_lens[bb]
        for h in range(4):
            g = h // 2
            ref = _sdpa(q[bb, h].astype(np.float64), _f64(k[bb, g, :Tb]), _f64(v[bb, g, :Tb]))
            np.testing.assert_allclose(r.o[bb, h], ref, rtol=1e-10, atol=1e-12)
            assert r.counts[bb, h] == Tb


def test_screen_all_is_dense_gated_attention():
    # softmax(S~) = softmax(S + (S~ - S)): SDPA with the gate's offset as an additive mask
    wl = make_workload(B=1, Hq=2, Hkv=1, d=16, block=8, seq_lens=[203], dtype=torch.float32,
                       predictor=False, tau_const=0.4, planted={"frac": 0.2}, seed=4)
    q, k, v = as_numpy(wl.q), as_numpy(wl.k), as_numpy(wl.v)
    tau = np.full((1, 2), 0.4)
    r = oracle.decode(q, k, v, wl.seq_lens, tau, block_size=8, beta=3.0, screen_all=True)
    for h in range(2):
        qh = q[0, h].astype(np.float64)
        S = _f64(k[0, 0]) @ qh / 4.0
        off = np.array([oracle.gate(s, 0.4, 3.0) - s for s in S])
        ref = _sdpa(qh, _f64(k[0, 0]), _f64(v[0, 0]), off)
        np.testing.assert_allclose(r.o[0, h], ref, rtol=1e-10, atol=1e-12)
        assert r.counts[0, h] == 203


def test_convex_output_decomposition():
    # o over a union of disjoint token sets is the Z-weighted combination of the parts
    rng = np.random.default_rng(8)
    T, b, d = 333, 16, 24
    K = rng.standard_normal((T, d)).astype(np.float32)
    V = rng.standard_normal((T, d)).astype(np.float32)
    q = rng.standard_normal(d)
    N = T // b
    for trial in range(5):
        part = rng.integers(0, 2, N).astype(np.uint8)
        o_all, l_all, n_all = oracle.attend(q, K, V, b, np.ones(N, np.uint8), use_tail=True,
                                            tau_eff=1.1, beta=4.0)
        o1, l1, n1 = oracle.attend(q, K, V, b, part, use_tail=False, tau_eff=1.1, beta=4.0)
        o2, l2, n2 = oracle.attend(q, K, V, b, 1 - part, use_tail=True, tau_eff=1.1, beta=4.0)
        Z1, Z2 = math.exp(l1) if n1 else 0.0, math.exp(l2)
        np.testing.assert_allclose(o_all, (Z1 * o1 + Z2 * o2) / (Z1 + Z2), rtol=1e-12, atol=1e-13)
        assert l_all == pytest.approx(math.log(Z1 + Z2), rel=1e-13)
        assert n_all == n1 + n2 == T


def test_nothing_attended_gives_zero_output():
    K = np.ones((32, 4), np.float32)
    o, lse, n = oracle.attend(np.ones(4), K, K, 16, np.zeros(2, np.uint8), use_tail=False)
    assert n == 0 and lse == -math.inf and np.all(o == 0)


def test_self_ungated_changes_only_the_last_key():
    rng = np.random.default_rng(1)
    K = rng.standard_normal((40, 8)).astype(np.float32)
    V = rng.standard_normal((40, 8)).astype(np.float32)
    q = rng.standard_normal(8)
    sel = np.ones(2, np.uint8)
    o0, l0, _ = oracle.attend(q, K, V, 16, sel, tau_eff=2.0, beta=4.0, self_ungated=False)
    o1, l1, _ = oracle.attend(q, K, V, 16, sel, tau_eff=2.0, beta=4.0, self_ungated=True)
    S_last = float(K[-1] @ q) / math.sqrt(8)
    g_last = oracle.gate(S_last, 2.0, 4.0)
    # closed-form swap of one weight: Z1 = Z0 - e^{g} + e^{S}
    Z0, Z1 = math.exp(l0), math.exp(l1)
    assert Z1 == pytest.approx(Z0 - math.exp(g_last) + math.exp(S_last), rel=1e-12)
    np.testing.assert_allclose(o1 * Z1, o0 * Z0 + (math.exp(S_last) - math.exp(g_last)) * V[-1].astype(np.float64),
                               rtol=1e-10, atol=1e-12)


# ------------------------------------------------------ whole path vs brute force

CASES = [
    # B, Hq, Hkv, d, b, lens, c, tau, z, a, lwb, self_ungated, dtype
    (1, 1, 1, 8, 4, [1], 4, 0.5, 1.0, 0.0, 0, False, torch.float32),
    (1, 1, 1, 8, 4, [3], 4, 0.5, 1.0, 0.0, 0, False, torch.float32),
    (1, 2, 1, 8, 4, [4], 4, 0.5, 1.0, 0.0, 0, False, torch.float32),
    (2, 2, 2, 8, 4, [37, 5], 3, 0.8, 1.0, 0.0, 0, True, torch.float32),
    (1, 4, 2, 16, 8, [100], 2, 3.0, 1.0, 0.0, 0, False, torch.float32),     # forces rescue
    (1, 4, 1, 16, 8, [100], 2, 3.0, 1.0, 0.0, 2, False, torch.float32),     # pins
    (2, 4, 2, 64, 16, [1024, 777], 16, 1.3, 2.0, 0.2, 0, False, torch.bfloat16),
    (1, 8, 2, 64, 64, [1000], 128, 1.5, 1.0, 0.0, 0, False, torch.bfloat16),
    (3, 4, 4, 8, 4, [64, 65, 66], 100, 0.2, 1.0, -0.3, 1, True, torch.bfloat16),
    (1, 2, 1, 32, 16, [512], 0, 5.0, 1.0, 0.0, 0, False, torch.float32),    # rescue off, tail-less
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_oracle_matches_brute_force_algorithm(case):
    B, Hq, Hkv, d, b, lens, c, tau0, z, a, lwb, su, dt = CASES[case]
    wl = make_workload(B=B, Hq=Hq, Hkv=Hkv, d=d, block=b, seq_lens=lens, dtype=dt,
                       predictor=False, tau_const=tau0, planted={"frac": 0.15}, seed=100 + case)
    q, k, v = as_numpy(wl.q), as_numpy(wl.k), as_numpy(wl.v)
    rng = np.random.default_rng(case)
    tau = tau0 + 0.3 * rng.standard_normal((B, Hq))
    r = oracle.decode(q, k, v, lens, tau, block_size=b, z=z, a=a, beta=4.0, rescue_window=c,
                      lwb=lwb, self_ungated=su)
    G = Hq // Hkv
    for bb in range(B):
        for h in range(Hq):
            o, att, ntok = brute.decode_head(q[bb, h], k[bb, h // G], v[bb, h // G], lens[bb], b, c,
                                             tau[bb, h], a=a, z=z, beta=4.0, lwb=lwb,
                                             self_ungated=su)
            np.testing.assert_allclose(r.o[bb, h], o, rtol=1e-10, atol=1e-12)
            assert set(np.nonzero(r.sel[bb, h])[0].tolist()) == att
            assert r.counts[bb, h] == ntok


# ----------------------------------------------------------- planted sanity

def test_config1_selects_exactly_the_planted_blocks():
    wl = config1()
    q, k, v = as_numpy(wl.q), as_numpy(wl.k), as_numpy(wl.v)
    tau = oracle.predict(q, None, as_numpy(wl.bias))
    assert np.all(tau == 2.0)
    r = oracle.decode(q, k, v, wl.seq_lens, tau, block_size=64, z=1.0, beta=4.0, rescue_window=128)
    for h in range(4):
        assert np.nonzero(r.sel[0, h])[0].tolist() == wl.planted[(0, h)].tolist()
        assert r.counts[0, h] == 8 * 64
        # planted scores ~ 3 |q| >> 0: the output is the planted-only attention
        o_p, _, _ = oracle.attend(q[0, h].astype(np.float64), k[0, h], v[0, h], 64, r.sel[0, h],
                                  use_tail=False, tau_eff=2.0, beta=4.0)
        np.testing.assert_allclose(r.o[0, h], o_p, rtol=1e-12)
    # the margin to the threshold is wide (no block inside the 1e-4 tie band)
    assert np.nanmin(np.abs(r.bounds - 2.0)) > 1e-2


def test_round_f16_is_ieee_binary16_nearest_even():
    """fp16 index records (App. "GQA-Grouped Execution and Compact Metadata Layout"):
    the oracle's rounding equals NumPy's float64 -> float16 conversion, an
    independent implementation of IEEE 754 round-to-nearest-even."""
    rng = np.random.default_rng(5)
    mag = 10.0 ** rng.uniform(-10, 6, 20000)
    x = np.concatenate([mag * rng.choice([-1.0, 1.0], mag.size),
                        rng.standard_normal(5000) * 3.0,
                        np.array([0.0, -0.0, np.inf, -np.inf, 65504.0, 65519.99, 65520.0, 7e4,
                                  2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -25, 2.0 ** -14,
                                  2.0 ** -14 - 2.0 ** -25])])
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).astype(np.float64)
    got = oracle.round_f16(x)
    assert np.array_equal(got, ref)
    assert np.array_equal(np.signbit(got), np.signbit(ref))
    assert np.isnan(oracle.round_f16([np.nan]))[0]
    # ties go to the even significand: 1 + 2^-11 -> 1, 1 + 3 * 2^-11 -> 1 + 2^-9,
    # half the smallest subnormal -> 0, 1.5 of it -> 2^-23
    assert oracle.round_f16([1 + 2.0 ** -11, 1 + 3 * 2.0 ** -11, 2.0 ** -25, 3 * 2.0 ** -25]).tolist() \
        == [1.0, 1 + 2.0 ** -9, 0.0, 2.0 ** -23]


def test_round_e4m3_is_fp8_nearest_even():
    """FP8 index records (Sec. "Limitations and Conclusion": FP8 metadata): on the
    finite range the oracle's rounding equals torch's float32 -> float8_e4m3fn
    conversion, an independent round-to-nearest-even implementation of the format;
    from 464 (the tie between 448 and the first step past it) it saturates to 448,
    where the format has no finite value and torch gives NaN."""
    rng = np.random.default_rng(6)
    mag = 2.0 ** rng.uniform(-13, np.log2(463.9), 20000)
    x = np.concatenate([mag * rng.choice([-1.0, 1.0], mag.size),
                        rng.standard_normal(5000) * 3.0,
                        np.array([0.0, -0.0, 448.0, 447.9, 463.9, -463.9, 2.0 ** -9, 2.0 ** -10,
                                  3 * 2.0 ** -10, 2.0 ** -6, 2.0 ** -6 - 2.0 ** -10, 1 + 2.0 ** -4,
                                  1 + 3 * 2.0 ** -4, 240.0 + 8.0, 256.0 + 16.0])])
    x = x.astype(np.float32)                          # exactly representable inputs
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = oracle.round_e4m3(x.astype(np.float64))
    assert np.array_equal(got, ref)
    assert np.array_equal(np.signbit(got), np.signbit(ref))
    assert np.isnan(oracle.round_e4m3([np.nan]))[0]
    assert oracle.round_e4m3([464.0, 480.0, 1e6, -500.0, np.inf]).tolist() == [448.0, 448.0, 448.0,
                                                                                -448.0, 448.0]
    # ties go to the even significand: 1 + 2^-4 -> 1, 1 + 3 * 2^-4 -> 1.25, half the
    # smallest subnormal -> 0, 1.5 of it -> 2^-8
    assert oracle.round_e4m3([1 + 2.0 ** -4, 1 + 3 * 2.0 ** -4, 2.0 ** -10, 3 * 2.0 ** -10]).tolist() \
        == [1.0, 1.25, 0.0, 2.0 ** -8]


# ------------------------------------------------------------- offline calibration
# App. "Offline Threshold Calibration via 1/t-Weighted Histograms",
# Alg. "Density-Matched Offline Threshold Calibration".

def _calib_inputs(seed, N=2, Hq=4, Hkv=2, T=40, d=8):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((N, Hq, T, d)).astype(np.float32)
    k = rng.standard_normal((N, Hkv, T, d)).astype(np.float32)
    return q, k


def test_calib_weights_sum_to_steps_and_brackets_order():
    q, k = _calib_inputs(1)
    N, Hq, T = q.shape[0], q.shape[1], q.shape[2]
    tau = np.random.default_rng(2).normal(0.5, 0.3, (N, Hq, T))
    r = oracle.calib_hist(q, k, tau, beta=4.0, lo=-3.0, hi=3.0, nb=64, gamma=1e-3, brackets=True)
    # sum over causal pairs of 1 / (steps seen) is one per step: N T per head
    np.testing.assert_allclose(r.total, N * T, rtol=1e-12)
    for H in (r.hist, r.hist_lo, r.hist_hi):
        np.testing.assert_allclose(H.sum(axis=1), N * T, rtol=1e-12)
    # binning at S - delta moves mass left, at S + delta right: cumulative sums bracket
    c, cl, ch = (np.cumsum(H, axis=1) for H in (r.hist, r.hist_lo, r.hist_hi))
    assert np.all(cl >= c - 1e-9) and np.all(c >= ch - 1e-9)
    assert np.all((r.target > 0) & (r.target < 1))


def test_calib_matches_brute_force_definition():
    """Tiny case, pure-Python loops over the definition of the weighted histogram
    and of the target density (causal pairs s <= t, weight 1/(t+1))."""
    q, k = _calib_inputs(3, N=2, Hq=2, Hkv=1, T=6, d=4)
    tau = np.random.default_rng(4).normal(0.0, 0.5, (2, 2, 6))
    lo, hi, nb, beta = -2.0, 2.0, 8, 3.0
    r = oracle.calib_hist(q, k, tau, beta=beta, lo=lo, hi=hi, nb=nb)
    w = (hi - lo) / nb
    for h in range(2):
        H = [0.0] * nb
        dens = 0.0
        for x in range(2):
            for t in range(6):
                for s in range(t + 1):
                    S = sum(float(q[x, h, t, i]) * float(k[x, 0, s, i]) for i in range(4)) / 2.0
                    b = min(max(int(math.floor((S - lo) / w)), 0), nb - 1)
                    H[b] += 1.0 / (t + 1)
                    dens += 1.0 / (1.0 + math.exp(-beta * (S - tau[x, h, t]))) / (t + 1)
        np.testing.assert_allclose(r.hist[h], H, rtol=1e-12, atol=1e-14)
        assert abs(r.dens[h] - dens) < 1e-12


def test_calib_constant_scores_closed_form():
    """q = 0 makes every score 0: all weight in the bin holding 0, whose centre is
    s0; with a constant dynamic threshold tau0 the target is sigmoid(-beta tau0),
    so g(c) = sigmoid(beta (s0 - c)) = target gives c = s0 + tau0 exactly."""
    q, k = _calib_inputs(5, N=1, Hq=2, Hkv=2, T=10, d=8)
    q[:] = 0.0
    lo, hi, nb = -1.0, 1.0, 10           # 0 lies in bin 5, centre 0.1
    for beta, tau0 in ((4.0, 0.3), (1.5, -0.8), (8.0, 2.0)):
        tau = np.full((1, 2, 10), tau0)
        r = oracle.calib_hist(q, k, tau, beta=beta, lo=lo, hi=hi, nb=nb)
        assert np.all(r.hist[:, 5] == r.total) and np.all(np.delete(r.hist, 5, axis=1) == 0)
        np.testing.assert_allclose(r.target, 1.0 / (1.0 + math.exp(beta * tau0)), rtol=1e-12)
        c = oracle.calib_solve(r.hist[0], lo, hi, beta, r.target[0])
        assert abs(c - (0.1 + tau0)) < 1e-12


def test_calib_g_monotone_and_constant_threshold_recovered():
    """g falls from 1 to 0; calibrating the densities a constant dynamic threshold
    realises returns that constant to within the bin width; the bisection residual
    is at rounding level (the paper's < 2e-16)."""
    q, k = _calib_inputs(6, N=2, Hq=4, Hkv=2, T=48, d=16)
    lo, hi, nb = -6.0, 6.0, 600
    for beta, tau0 in ((4.0, 0.7), (2.0, -0.5), (6.0, 1.6)):
        tau = np.full((2, 4, 48), tau0)
        r = oracle.calib_hist(q, k, tau, beta=beta, lo=lo, hi=hi, nb=nb)
        for h in range(4):
            cs = np.linspace(lo - 10, hi + 10, 200)
            g = np.array([oracle.calib_g(r.hist[h], lo, hi, beta, c) for c in cs])
            inner = (g[:-1] > 1e-12) & (g[:-1] < 1 - 1e-12)
            assert np.all(np.diff(g) <= 0) and np.all(np.diff(g)[inner] < 0)
            assert g[0] > 1 - 1e-9 and g[-1] < 1e-9
            c = oracle.calib_solve(r.hist[h], lo, hi, beta, r.target[h])
            assert abs(c - tau0) <= (hi - lo) / nb, (beta, tau0, h, c)
            assert abs(oracle.calib_g(r.hist[h], lo, hi, beta, c) - r.target[h]) < 1e-15


# ------------------------------------------------------------- gated prefill forward
# App. "Hardware-Aligned Forward Kernel" (Alg. fwd_kernel).

def _prefill_inputs(seed, B=2, Hq=4, Hkv=2, T=24, d=16):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, Hq, T, d)).astype(np.float32)
    k = rng.standard_normal((B, Hkv, T, d)).astype(np.float32)
    v = rng.standard_normal((B, Hkv, T, d)).astype(np.float32)
    return q, k, v


def _expand_kv(x, G):
    return np.repeat(x, G, axis=1)


def test_prefill_ungated_is_causal_softmax_attention():
    """tau = -inf: every gate is 1, so O is causal softmax attention (torch SDPA in
    fp64), L its log-sum-exp, R_i = i + 1; rows past a sequence's length are empty."""
    q, k, v = _prefill_inputs(11)
    B, Hq, T, d = q.shape
    G = Hq // k.shape[1]
    r = oracle.prefill(q, k, v, np.full((B, Hq, T), -np.inf), [T, 17], beta=4.0)
    qt = torch.tensor(q, dtype=torch.float64)
    kt = torch.tensor(_expand_kv(k, G), dtype=torch.float64)
    vt = torch.tensor(_expand_kv(v, G), dtype=torch.float64)
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True).numpy()
    S = (qt @ kt.transpose(-1, -2)) / math.sqrt(d)
    S = S.masked_fill(torch.triu(torch.ones(T, T, dtype=torch.bool), 1), float("-inf"))
    lse = torch.logsumexp(S, dim=-1).numpy()
    np.testing.assert_allclose(r.o[0], ref[0], atol=1e-12)
    np.testing.assert_allclose(r.lse[0], lse[0], atol=1e-12)
    np.testing.assert_allclose(r.o[1, :, :17], ref[1, :, :17], atol=1e-12)
    np.testing.assert_array_equal(r.r[0], np.broadcast_to(np.arange(1, T + 1), (Hq, T)))
    assert np.all(r.o[1, :, 17:] == 0) and np.all(np.isneginf(r.lse[1, :, 17:]))
    assert np.all(r.r[1, :, 17:] == 0)


def test_prefill_closed_gates_leave_only_the_diagonal():
    """tau = +inf: every gate is 0.  Multiplicative: S~ = 0 off the diagonal and S_ii on
    it, so O_i = (sum_{j<i} v_j + e^{S_ii} v_i) / (i + e^{S_ii}).  Additive with C:
    S~ = S - C off the diagonal.  R = 0."""
    q, k, v = _prefill_inputs(12, B=1, Hq=2, Hkv=1, T=12, d=8)
    T, d = 12, 8
    tau = np.full((1, 2, T), np.inf)
    r = oracle.prefill(q, k, v, tau, [T], beta=3.0)
    ra = oracle.prefill(q, k, v, tau, [T], beta=3.0, additive=True, C=2.5)
    kv, vv = k[0, 0].astype(np.float64), v[0, 0].astype(np.float64)
    for h in range(2):
        qq = q[0, h].astype(np.float64)
        for i in range(T):
            sii = float(qq[i] @ kv[i]) / math.sqrt(d)
            e = math.exp(sii)
            want = (vv[:i].sum(axis=0) + e * vv[i]) / (i + e)
            np.testing.assert_allclose(r.o[0, h, i], want, atol=1e-12)
            s = np.array([float(qq[i] @ kv[j]) / math.sqrt(d) - 2.5 for j in range(i)] + [sii])
            w = np.exp(s - s.max())
            np.testing.assert_allclose(ra.o[0, h, i], (w[:, None] * vv[:i + 1]).sum(0) / w.sum(),
                                       atol=1e-12)
    assert np.all(r.r == 0)


def test_prefill_last_row_is_dense_gated_decode():
    """The prefill's last row is the decode step at the same position over every
    key with the gate (screen_all) and the diagonal bypass (self_ungated): two
    independently written routines of the oracle."""
    q, k, v = _prefill_inputs(13, B=2, Hq=4, Hkv=2, T=64, d=16)
    tau = np.random.default_rng(14).normal(0.3, 0.5, (2, 4, 64))
    r = oracle.prefill(q, k, v, tau, [64, 64], beta=4.0)
    dec = oracle.decode(np.ascontiguousarray(q[:, :, -1]), k, v, [64, 64], tau[:, :, -1],
                        block_size=16, beta=4.0, z=1.0, rescue_window=0, screen_all=True,
                        self_ungated=True)
    np.testing.assert_allclose(r.o[:, :, -1], dec.o, atol=1e-12)
    np.testing.assert_allclose(r.lse[:, :, -1], dec.lse, atol=1e-12)


def test_prefill_matches_brute_force_definition():
    q, k, v = _prefill_inputs(15, B=1, Hq=2, Hkv=1, T=7, d=4)
    tau = np.random.default_rng(16).normal(0.0, 0.7, (1, 2, 7))
    beta, C = 2.5, 1.7
    for additive in (False, True):
        r = oracle.prefill(q, k, v, tau, [7], beta=beta, additive=additive, C=C)
        for h in range(2):
            for i in range(7):
                sc, gs = [], 0.0
                for j in range(i + 1):
                    S = sum(float(q[0, h, i, c]) * float(k[0, 0, j, c]) for c in range(4)) / 2.0
                    g = 1.0 / (1.0 + math.exp(-beta * (S - tau[0, h, i])))
                    gs += g
                    sc.append(S if j == i else (S + C * g - C if additive else S * g))
                mx = max(sc)
                w = [math.exp(x - mx) for x in sc]
                o = [sum(w[j] * float(v[0, 0, j, c]) for j in range(i + 1)) / sum(w) for c in range(4)]
                np.testing.assert_allclose(r.o[0, h, i], o, atol=1e-12)
                assert abs(r.r[0, h, i] - gs) < 1e-12
                assert abs(r.lse[0, h, i] - (mx + math.log(sum(w)))) < 1e-12


def test_prefill_rows_are_the_full_rows():
    """prefill_rows (sampled rows of long sequences) returns exactly the rows of the
    pinned full forward, rows past a sequence's length included."""
    q, k, v = _prefill_inputs(17, B=2, Hq=4, Hkv=2, T=40, d=16)
    tau = np.random.default_rng(18).normal(0.2, 0.5, (2, 4, 40))
    for additive in (False, True):
        full = oracle.prefill(q, k, v, tau, [40, 23], beta=3.0, additive=additive, C=1.5)
        rows = np.array([[0, 0, 0], [0, 3, 39], [1, 2, 22], [1, 1, 23], [1, 0, 39], [0, 1, 17]])
        r = oracle.prefill_rows(q, k, v, tau, [40, 23], rows, beta=3.0, additive=additive, C=1.5)
        for n, (b, h, i) in enumerate(rows):
            np.testing.assert_array_equal(r.o[n], full.o[b, h, i])
            assert r.r[n] == full.r[b, h, i] and r.lse[n] == full.lse[b, h, i]


# --------------------------------------------------------------------- screening quality
#
# The diagnostics of Tab. "index_quality": block false negatives / positives,
# recall of above-threshold keys and the missed gated softmax mass.

def _quality_keys():
    """d = 4, b = 2 (scale 1/2 exact), q = (2, 0, 0, 0): each key's score is its first
    coordinate exactly.  Block 0 = keys -1, 3 (maximum at its last key), block 1 =
    keys 1, 0.2 (maximum exactly at tau = 1), tail = one key of score 1."""
    k = np.zeros((5, 4), np.float32)
    k[:, 0] = [-1.0, 3.0, 1.0, 0.2, 1.0]
    return np.array([2.0, 0.0, 0.0, 0.0]), k


def test_screen_quality_hand_worked_example():
    q, k = _quality_keys()
    S = [-1.0, 3.0, 1.0, float(np.float32(0.2)), 1.0]
    g = [oracle.gate(s, 1.0, 4.0) for s in S]           # the gate is pinned above
    m = max(g)
    w = [math.exp(x - m) for x in g]
    Z = sum(w)
    # block 0 selected: block 1 (maximum 1 >= tau) is a false negative; of the two
    # above-threshold keys of the full blocks (3 and 1; the tail's is not screened)
    # one is attended; the missed mass is block 1's share of all five keys
    r = oracle.screen_quality(q, k, 2, [1, 0], tau_eff=1.0, beta=4.0)
    assert (r["positive_blocks"], r["false_negative_blocks"], r["false_positive_blocks"],
            r["selected_blocks"], r["above_keys"], r["above_keys_attended"]) == (2, 1, 0, 1, 2, 1)
    np.testing.assert_array_equal(r["blockmax"], [3.0, 1.0])
    assert r["missed_mass"] == pytest.approx((w[2] + w[3]) / Z, rel=1e-14)
    # block 1 selected instead: block 0 is the false negative
    r = oracle.screen_quality(q, k, 2, [0, 1], tau_eff=1.0, beta=4.0)
    assert (r["false_negative_blocks"], r["above_keys_attended"]) == (1, 1)
    assert r["missed_mass"] == pytest.approx((w[0] + w[1]) / Z, rel=1e-14)
    # nothing selected: both blocks missed, only the tail's mass kept
    r = oracle.screen_quality(q, k, 2, [0, 0], tau_eff=1.0, beta=4.0)
    assert (r["false_negative_blocks"], r["above_keys_attended"]) == (2, 0)
    assert r["missed_mass"] == pytest.approx(1.0 - w[4] / Z, rel=1e-14)
    # threshold above every score: no positive block, a selected block is a false positive
    r = oracle.screen_quality(q, k, 2, [1, 1], tau_eff=3.5, beta=4.0)
    assert (r["positive_blocks"], r["false_positive_blocks"], r["above_keys"]) == (0, 2, 0)
    assert r["missed_mass"] == 0.0


def _quality_workload(seed=3):
    return make_workload(B=2, Hq=4, Hkv=2, d=32, block=16, seq_lens=[1000, 611], dtype=torch.float32,
                         planted={"frac": 0.1}, predictor=False, tau_const=1.2, seed=seed)


def test_blockmax_is_brute_force_maximum():
    wl = _quality_workload()
    q, k, v = (as_numpy(t) for t in (wl.q, wl.k, wl.v))
    tau = np.full((2, 4), 1.2)
    r = oracle.decode(q, k, v, wl.seq_lens, tau, block_size=16, z=1.0, quality=True)
    for b in range(2):
        N = wl.seq_lens[b] // 16
        for h in range(4):
            S = (k[b, h // 2, :N * 16].astype(np.float64) @ q[b, h].astype(np.float64)) / math.sqrt(32)
            np.testing.assert_allclose(r.blockmax[b, h, :N], S.reshape(N, 16).max(axis=1), rtol=1e-13)
            above = S >= 1.2
            sel = np.repeat(r.sel[b, h, :N].astype(bool), 16)
            assert r.quality[b, h, 4] == above.sum() and r.quality[b, h, 5] == (above & sel).sum()


def test_missed_mass_is_the_log_sum_exp_gap():
    """The attended set and the rejected blocks partition the keys, so the rejected
    share of the dense gated mass is 1 - exp(lse_attended - lse_all) (the convex
    decomposition of the output over a partition)."""
    wl = _quality_workload(seed=5)
    q, k, v = (as_numpy(t) for t in (wl.q, wl.k, wl.v))
    tau = np.array([[1.0, 1.5, 2.0, 0.5], [1.2, 0.8, 2.5, 1.7]])
    r = oracle.decode(q, k, v, wl.seq_lens, tau, block_size=16, z=1.0, quality=True)
    full = oracle.decode(q, k, v, wl.seq_lens, tau, block_size=16, z=1.0, screen_all=True)
    gap = 1.0 - np.exp(r.lse - full.lse)
    np.testing.assert_allclose(r.missed, gap, rtol=1e-9, atol=1e-14)
    assert np.all(r.missed > 0.0)


@pytest.mark.parametrize("b,d", [(16, 32), (64, 64)])
def test_no_false_negatives_at_the_certified_z(b, d):
    """At z = sqrt((b - 1) d) the dual bound is at least every block's maximum score
    (Samuelson + Cauchy-Schwarz), so every positive block is selected."""
    wl = make_workload(B=1, Hq=4, Hkv=1, d=d, block=b, seq_lens=[b * 40], dtype=torch.float32,
                       planted={"frac": 0.1}, predictor=False, tau_const=0.0, seed=b + d)
    q, k, v = (as_numpy(t) for t in (wl.q, wl.k, wl.v))
    r0 = oracle.decode(q, k, v, wl.seq_lens, np.zeros((1, 4)), block_size=b, z=1.0, quality=True,
                       rescue_window=0)
    tau = np.median(r0.blockmax[0], axis=1)[None, :]      # about half the blocks positive
    zc = math.sqrt((b - 1) * d)
    r = oracle.decode(q, k, v, wl.seq_lens, tau, block_size=b, z=zc, quality=True, rescue_window=0)
    assert np.all(r.quality[0, :, 0] > 0)
    assert np.all(r.quality[0, :, 1] == 0) and np.all(r.quality[0, :, 4] == r.quality[0, :, 5])
    # not vacuous: without the z term the same blocks are missed
    r = oracle.decode(q, k, v, wl.seq_lens, tau, block_size=b, z=0.0, quality=True, rescue_window=0)
    assert r.quality[0, :, 1].sum() > 0


def test_quality_of_screen_all_and_open_threshold():
    wl = _quality_workload(seed=7)
    q, k, v = (as_numpy(t) for t in (wl.q, wl.k, wl.v))
    tau = np.full((2, 4), 1.2)
    r = oracle.decode(q, k, v, wl.seq_lens, tau, block_size=16, z=1.0, quality=True, screen_all=True)
    rates = oracle.quality_rates(r)
    assert rates["false_negative_rate"] == 0.0 and rates["token_recall"] == 1.0
    assert rates["missed_mass_max"] == 0.0
    for b in range(2):
        N = wl.seq_lens[b] // 16
        assert np.all(r.quality[b, :, 2] == N - r.quality[b, :, 0])
    r = oracle.decode(q, k, v, wl.seq_lens, np.full((2, 4), -np.inf), block_size=16, z=1.0,
                      quality=True)
    for b in range(2):
        N = wl.seq_lens[b] // 16
        assert np.all(r.quality[b, :, 0] == N) and np.all(r.quality[b, :, 1] == 0)
    assert np.all(r.missed == 0.0)
