"""GPU parity of the block-index variants: the sub-block variance envelope and
the incremental decode-time update (needs an MI355X).

  * envelope sigma against the oracle's Eq. (subblock_envelope_appx) for every
    (head dim, block, dtype) kernel shape and sub-block lengths below, equal to
    and above the rows one load covers; mu and M are the flat build's, bit for
    bit; sub_block = block_size reproduces the flat sigma bit for bit;
  * the update writes exactly the records of the blocks completed since
    prev_lens (capped at max_new_blocks), equal bit for bit to a full build,
    and leaves every other entry alone; a token-by-token decode loop ends with
    the full build's index;
  * a decode step on envelope summaries matches the oracle run on the oracle's
    own envelope summaries.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_support import (calibrate_bias, compare, oracle_inputs, oracle_summaries, require_gpu,
                         run_gpu, run_oracle, say)
from paper_2609_20888_amd import eta
from synth import as_numpy, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(request):
    require_gpu()
    say(f"\n[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


def _np(s: eta.Summaries):
    return s.mu.cpu().numpy(), s.sigma.cpu().numpy(), s.max_norm.cpu().numpy()


ENVELOPE_CASES = [
    # B, Hkv, d, b, lens, dtype, sub_blocks
    (1, 2, 128, 64, [64 * 40 + 9], torch.bfloat16, (1, 2, 4, 8, 16)),
    (1, 1, 128, 128, [128 * 35], torch.bfloat16, (4, 32)),
    (2, 1, 64, 64, [64 * 33, 64 * 7 + 1], torch.bfloat16, (2, 4, 8, 16)),
    (1, 1, 64, 128, [128 * 20], torch.bfloat16, (4, 64)),
    (1, 1, 128, 64, [64 * 30], torch.float32, (1, 4, 16)),
    (1, 1, 64, 64, [64 * 30], torch.float32, (2, 4, 32)),
]


@pytest.mark.parametrize("case", range(len(ENVELOPE_CASES)))
def test_envelope_matches_oracle(case):
    B, Hkv, d, b, lens, dt, subs = ENVELOPE_CASES[case]
    wl = make_workload(B=B, Hq=Hkv, Hkv=Hkv, d=d, block=b, seq_lens=lens, dtype=dt,
                       planted={"frac": 0.1}, predictor=False, tau_const=1.0, seed=40 + case)
    dev = torch.device("cuda")
    k = wl.k.to(dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    fmu, fsg, fmx = _np(eta.build_block_summaries(k, sl, b))
    kn = as_numpy(wl.k)
    for sub in subs:
        mu, sg, mx = _np(eta.build_block_summaries(k, sl, b, sub_block=sub))
        for bb in range(B):
            N = lens[bb] // b
            np.testing.assert_array_equal(mu[bb, :, :, :N], fmu[bb, :, :, :N])
            np.testing.assert_array_equal(mx[bb, :, :N], fmx[bb, :, :N])
            for g in range(Hkv):
                omu, _, _ = oracle.summaries(kn[bb, g, :lens[bb]], b)
                env = oracle.envelope(kn[bb, g, :lens[bb]], b, sub, omu)
                np.testing.assert_allclose(sg[bb, g, :, :N].T, env, rtol=1e-5, atol=1e-5,
                                           err_msg=f"sub_block {sub}")
                # the envelope dominates the flat sigma up to rounding (mean of sub-block MSDs <= max)
                assert np.all(sg[bb, g, :, :N] >= fsg[bb, g, :, :N] * (1 - 1e-5) - 1e-6)


@pytest.mark.parametrize("d,b,dt", [(128, 128, torch.bfloat16), (64, 64, torch.bfloat16),
                                    (128, 64, torch.float32)])
def test_envelope_of_one_sub_block_is_flat_sigma(d, b, dt):
    wl = make_workload(B=1, Hq=2, Hkv=2, d=d, block=b, seq_lens=[b * 50 + 3], dtype=dt,
                       planted={"frac": 0.1}, predictor=False, tau_const=1.0, seed=47)
    dev = torch.device("cuda")
    k = wl.k.to(dev)
    sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
    flat = _np(eta.build_block_summaries(k, sl, b))
    env = _np(eta.build_block_summaries(k, sl, b, sub_block=b))
    N = wl.seq_lens[0] // b
    for x, y in zip(flat, env):
        np.testing.assert_array_equal(x[..., :N], y[..., :N])


def _sentinel(B, Hkv, d, ncap, dev):
    s = eta.Summaries.empty(B, Hkv, d, ncap, dev)
    for t in (s.mu, s.sigma, s.max_norm):
        t.fill_(float("nan"))
    return s


UPDATE_CASES = [
    # d, b, dtype, prev lens, new lens, max_new_blocks, sub_block
    (128, 128, torch.bfloat16, [128 * 30 + 127, 128 * 9], [128 * 31, 128 * 9 + 5], 1, 0),
    (128, 64, torch.bfloat16, [64 * 20 + 3, 64 * 5, 0], [64 * 23 + 1, 64 * 5 + 63, 64 * 2], 3, 0),
    (128, 64, torch.bfloat16, [64 * 20 + 3, 64 * 40], [64 * 23 + 1, 64 * 35], 2, 0),     # cap; shrink
    (64, 64, torch.float32, [64 * 10], [64 * 50 + 7], 64, 4),                              # > 32 blocks
    (64, 128, torch.bfloat16, [128 * 3 + 1], [128 * 4], 1, 8),
]


@pytest.mark.parametrize("case", range(len(UPDATE_CASES)))
def test_update_writes_exactly_the_completed_blocks(case):
    d, b, dt, prev, new, max_new, sub = UPDATE_CASES[case]
    B, Hkv = len(prev), 2
    T_cap = b * 64
    wl = make_workload(B=B, Hq=4, Hkv=Hkv, d=d, block=b, seq_lens=[T_cap] * B, T_cap=T_cap,
                       dtype=dt, planted={"frac": 0.1}, predictor=False, tau_const=1.0,
                       seed=50 + case)
    dev = torch.device("cuda")
    k = wl.k.to(dev)
    pl = torch.tensor(prev, dtype=torch.int32, device=dev)
    nl = torch.tensor(new, dtype=torch.int32, device=dev)
    ncap = T_cap // b
    full = _np(eta.build_block_summaries(k, nl, b, sub_block=sub))
    s = eta.build_block_summaries(k, pl, b, sub_block=sub, out=_sentinel(B, Hkv, d, ncap, dev))
    before = _np(s)
    eta.update_block_summaries(k, pl, nl, s, b, max_new_blocks=max_new, sub_block=sub)
    after = _np(s)
    for bb in range(B):
        p_n, n_n = prev[bb] // b, new[bb] // b
        hi = min(n_n, p_n + max_new)
        written = np.zeros(ncap, bool)
        written[p_n:max(hi, p_n)] = True
        for x_full, x_before, x_after in zip(full, before, after):
            xa = np.moveaxis(x_after[bb], -1, 0) if x_after.ndim == 4 else x_after[bb].T
            xb = np.moveaxis(x_before[bb], -1, 0) if x_before.ndim == 4 else x_before[bb].T
            xf = np.moveaxis(x_full[bb], -1, 0) if x_full.ndim == 4 else x_full[bb].T
            # block axis first
            np.testing.assert_array_equal(xa[written], xf[written])
            np.testing.assert_array_equal(xa[~written], xb[~written])
        say(f"[gpu] seq {bb}: blocks {p_n}..{hi - 1} written")


@pytest.mark.parametrize("sub", [0, 4])
def test_token_by_token_decode_loop_rebuilds_the_index(sub):
    d, b = 128, 64
    L0, steps = 64 * 6 + 50, 3 * 64 + 20
    wl = make_workload(B=2, Hq=8, Hkv=2, d=d, block=b, seq_lens=[L0 + steps, L0 + steps],
                       T_cap=L0 + steps + 64, planted={"frac": 0.1}, predictor=False,
                       tau_const=1.0, seed=60)
    dev = torch.device("cuda")
    k = wl.k.to(dev)
    lens = torch.tensor([L0, L0 - 30], dtype=torch.int32, device=dev)
    s = eta.build_block_summaries(k, lens, b, sub_block=sub)
    for _ in range(steps):
        prev = lens.clone()
        lens += 1
        eta.update_block_summaries(k, prev, lens, s, b, max_new_blocks=1, sub_block=sub)
    ref = _np(eta.build_block_summaries(k, lens, b, sub_block=sub))
    got = _np(s)
    for bb in range(2):
        N = int(lens[bb]) // b
        for x, y in zip(got, ref):
            np.testing.assert_array_equal(x[bb, ..., :N], y[bb, ..., :N])


@pytest.mark.parametrize("sub,lwb", [(4, 2), (16, 0)])
def test_decode_on_envelope_summaries_matches_oracle(sub, lwb):
    wl = make_workload(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[20000, 9001],
                       planted={"frac": 0.05}, predictor=False, tau_const=2.0, lwb=lwb,
                       seed=70 + sub)
    np_in = oracle_inputs(wl)
    calibrate_bias(wl, np_in)
    g = run_gpu(wl, sub_block=sub)
    summ = oracle_summaries(wl, np_in[1], sub_block=sub)
    orc, tau_o = run_oracle(wl, np_in, summaries=summ)
    stats = compare(wl, g, orc, tau_o, np_inputs=np_in, union_counts=g.union_counts)
    frac = float(g.mask.float().mean())
    say(f"[gpu] envelope sub {sub} lwb {lwb}: {stats}, mask density {frac:.3f}")
