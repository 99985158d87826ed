"""Host logic of the synthetic workloads (CPU only): the predictor-bias placement."""
import numpy as np

from synth import place_bias


def test_place_bias_gives_the_target_survival_per_head_over_a_batch():
    # per-sequence predictor outputs much wider than the bounds' spread
    rng = np.random.default_rng(3)
    B, Hq, N = 8, 4, 512
    bounds = rng.normal(1.0, 0.125, (B, Hq, N))
    qW = rng.normal(0.0, 0.9, (B, Hq))
    for target in (0.01, 0.1, 0.2, 0.5):
        bias = place_bias(bounds, [N] * B, qW, target, a=0.25).astype(np.float64)
        tau_eff = qW[:, :, None] + bias[None, :, None] - 0.25
        kept = (bounds >= tau_eff).sum(axis=(0, 2))
        assert np.all(kept == int(np.ceil(target * B * N))), (target, kept)
        # no bound within 1e-6 of its threshold
        assert np.min(np.abs(bounds - tau_eff)) > 1e-6


def test_place_bias_ragged_lengths_ignore_blocks_past_the_end():
    rng = np.random.default_rng(4)
    B, Hq, Ncap = 3, 2, 100
    nblk = [100, 37, 5]
    bounds = rng.normal(0.0, 1.0, (B, Hq, Ncap))
    for b in range(B):
        bounds[b, :, nblk[b]:] = 1e9          # not full blocks: must not count
    qW = rng.normal(0.0, 0.5, (B, Hq))
    bias = place_bias(bounds, nblk, qW, 0.3).astype(np.float64)
    for h in range(Hq):
        kept = sum(int(np.sum(bounds[b, h, :nblk[b]] >= qW[b, h] + bias[h])) for b in range(B))
        assert kept == int(np.ceil(0.3 * sum(nblk)))
