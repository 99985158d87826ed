"""GPU parity of the offline density-matched calibration (App. "Offline Threshold
Calibration via 1/t-Weighted Histograms"; Alg. "Density-Matched Offline
Threshold Calibration"); needs an MI355X.

The GPU computes scores on the matrix cores in fp32 and bins them in fp32; a
score within its error bound of a bin edge may land in the next bin.  The
oracle therefore also bins every pair at S - delta and S + delta with
  delta = d 2^-24 sum_i |q_i k_i| / sqrt(d) + 8 2^-24 (|lo| + |hi| + S_max)
(the classical bound for d fp32 additions of exact products, plus the binning
arithmetic; S_max = max |q| max |k| / sqrt(d) by Cauchy-Schwarz), and the
GPU's cumulative histogram must lie between those two.  The target densities
agree to the gate's slope (beta / 4) times the largest delta; the constants
solve the oracle's equation g(c) = target up to the change that moving the
ambiguous mass to a neighbouring bin can make in g (beta w / 4 per unit of
mass).  Accumulation is in integers, so it is exactly reproducible and
additive over calls.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from gpu_support import require_gpu, say
from paper_2609_20888_amd import eta
from synth import as_numpy, calib_stream

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


@pytest.fixture(autouse=True)
def _gpu(request):
    require_gpu()
    say(f"\n[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


def _gpu_calibrate(cs, *, beta, lo, hi, nb, splits=1):
    Hq, Hkv, d = cs.q.shape[1], cs.k.shape[1], cs.q.shape[3]
    cal = eta.Calibrator(Hq, Hkv, d, beta=beta, lo=lo, hi=hi, num_bins=nb, device="cuda")
    N = cs.q.shape[0]
    cuts = np.linspace(0, N, splits + 1).astype(int)
    for a, b in zip(cuts[:-1], cuts[1:]):
        cal.accumulate(cs.q[a:b].contiguous(), cs.k[a:b].contiguous(), cs.tau[a:b].contiguous())
    c, target = cal.solve()
    torch.cuda.synchronize()
    hist = cal.hist.cpu().numpy().view(np.uint64)
    dens = cal.density.cpu().numpy().view(np.uint64)
    return hist, dens, c.cpu().numpy(), target.cpu().numpy()


CASES = [
    # N, Hq, Hkv, T, d, beta, lo, hi, nb
    (3, 8, 2, 200, 128, 4.0, -4.0, 8.0, 256),
    (2, 4, 4, 77, 64, 2.0, -3.0, 6.0, 1024),
    (1, 8, 1, 33, 128, 8.0, -5.0, 10.0, 64),
    (2, 16, 2, 130, 128, 4.0, -2.0, 2.0, 4096),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_calibration_matches_oracle(case):
    N, Hq, Hkv, T, d, beta, lo, hi, nb = CASES[case]
    cs = calib_stream(N=N, Hq=Hq, Hkv=Hkv, T=T, d=d, seed=100 + case, device="cuda")
    hist, dens, c, target = _gpu_calibrate(cs, beta=beta, lo=lo, hi=hi, nb=nb)
    qn, kn = as_numpy(cs.q), as_numpy(cs.k)
    tau = cs.tau.cpu().numpy().astype(np.float64)
    s_max = float(cs.q.float().norm(dim=-1).max() * cs.k.float().norm(dim=-1).max()) / math.sqrt(d)
    eps_abs = 8 * U * (abs(lo) + abs(hi) + s_max)
    delta_max = d * U * s_max + eps_abs
    r = oracle.calib_hist(qn, kn, tau, beta=beta, lo=lo, hi=hi, nb=nb, gamma=d * U,
                          eps_abs=eps_abs, brackets=True)
    H = hist.astype(np.float64) / eta.CALIB_UNIT
    total = N * T
    # weights: one per step, up to the fixed-point rounding of each 1/(t+1)
    np.testing.assert_allclose(H.sum(axis=1), r.total, rtol=0, atol=1e-6)
    cg, cl, ch = np.cumsum(H, axis=1), np.cumsum(r.hist_lo, axis=1), np.cumsum(r.hist_hi, axis=1)
    assert np.all(cg <= cl + 1e-6) and np.all(cg >= ch - 1e-6)
    amb = (cl - ch).sum(axis=1) / total                    # mass that may sit one bin over
    w = (hi - lo) / nb
    # target density: gate slope <= beta / 4 times the score error; fp32 gate rounding
    tgt_tol = beta / 4 * delta_max + 1e-6
    np.testing.assert_allclose(target, r.target, rtol=0, atol=tgt_tol)
    np.testing.assert_allclose(dens.astype(np.float64) / eta.CALIB_UNIT / total, r.target, atol=tgt_tol)
    worst = 0.0
    for h in range(Hq):
        resid = abs(oracle.calib_g(r.hist[h], lo, hi, beta, float(c[h])) - r.target[h])
        tol = amb[h] * beta * w / 4 + tgt_tol + beta / 4 * abs(float(c[h])) * U + 1e-9
        assert resid <= tol, (h, resid, tol)
        worst = max(worst, resid)
    c_orc = np.array([oracle.calib_solve(r.hist[h], lo, hi, beta, r.target[h]) for h in range(Hq)])
    say(f"[gpu] calibration case {case}: max |c_gpu - c_oracle| {np.max(np.abs(c - c_orc)):.2e}, "
        f"max g residual {worst:.2e}, ambiguous mass {amb.max():.2e}")


def test_calibration_is_reproducible_and_additive():
    cs = calib_stream(N=4, Hq=8, Hkv=2, T=150, d=128, seed=7, device="cuda")
    kw = dict(beta=4.0, lo=-4.0, hi=8.0, nb=512)
    a = _gpu_calibrate(cs, **kw)
    b = _gpu_calibrate(cs, **kw)
    c = _gpu_calibrate(cs, splits=3, **kw)
    for x, y, z in zip(a, b, c):
        assert np.array_equal(x, y) and np.array_equal(x, z)


def test_constant_dynamic_threshold_is_recovered():
    """Calibrating a predictor that always outputs tau0_h returns tau0_h to within a bin."""
    tau0 = [0.25 * h - 0.5 for h in range(8)]
    cs = calib_stream(N=2, Hq=8, Hkv=2, T=256, d=128, seed=8, tau_const=tau0, device="cuda")
    lo, hi, nb = -6.0, 10.0, 4096
    _, _, c, _ = _gpu_calibrate(cs, beta=4.0, lo=lo, hi=hi, nb=nb)
    assert np.all(np.abs(c - np.array(tau0)) <= (hi - lo) / nb), c
