"""GPU parity of the FP8 block index (8-bit E4M3 mu / sigma records, fp32 M;
FP8 metadata quantisation, Sec. "Limitations and Conclusion"); needs an MI355X.

  * the FP8 records are the fp32 statistics rounded to the nearest E4M3 value
    (ties to even, saturating at +-448), bit for bit (self-consistency with the
    fp32 build, rounded by the oracle's own oracle.round_e4m3); each lies in the
    interval of E4M3 values that rounding any fp32 statistic within the
    summation error bound of the oracle's fp64 one can give
    (gpu_support.f16_record_ranges with the E4M3 rounding); M is the fp32
    build's;
  * statistics that the fp32 build computes exactly (constant and two-valued
    key columns) land on E4M3's edge cases: ties in the normal and subnormal
    ranges, the smallest normal, carries into the next binade, and
    saturation; their codes are oracle.round_e4m3 of the exact statistic;
  * the incremental update writes the same FP8 codes as a full build;
  * a decode step screening on FP8 records matches the oracle screening on its
    own E4M3-rounded records, with the tie band widened by the largest bound
    change the record intervals allow (gpu_support.f16_band).
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_support import (calibrate_bias, compare, f16_band, f16_record_ranges, oracle_inputs,
                         oracle_summaries, require_gpu, run_gpu, run_oracle, say)
from paper_2609_20888_amd import eta
from synth import as_numpy, make_workload

pytestmark = pytest.mark.gpu

FP8 = torch.float8_e4m3fn


@pytest.fixture(autouse=True)
def _gpu(request):
    require_gpu()
    say(f"\n[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


def _f64(t: torch.Tensor) -> np.ndarray:
    """Record tensor (any of the three formats) as float64 on the CPU."""
    return t.detach().cpu().float().numpy().astype(np.float64)


FP8_CASES = [
    # Hkv, d, b, lens, dtype, sub_block
    (2, 128, 128, [128 * 60 + 5], torch.bfloat16, 0),
    (2, 128, 64, [64 * 70, 64 * 3 + 1], torch.bfloat16, 0),
    (1, 64, 64, [64 * 40], torch.float32, 0),
    (2, 128, 64, [64 * 50 + 7], torch.bfloat16, 4),
]


@pytest.mark.parametrize("case", range(len(FP8_CASES)))
def test_fp8_records_are_rounded_statistics(case):
    Hkv, d, b, lens, dt, sub = FP8_CASES[case]
    B = len(lens)
    wl = make_workload(B=B, Hq=Hkv, Hkv=Hkv, d=d, block=b, seq_lens=lens, dtype=dt,
                       planted={"frac": 0.1}, predictor=False, tau_const=1.0, seed=180 + case)
    dev = torch.device("cuda")
    k = wl.k.to(dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    s32 = eta.build_block_summaries(k, sl, b, sub_block=sub)
    s8 = eta.build_block_summaries(k, sl, b, sub_block=sub, stat_dtype=FP8)
    torch.cuda.synchronize()
    assert s8.mu.dtype == FP8 and s8.max_norm.dtype == torch.float32
    assert s8.mu.element_size() == 1
    kn = as_numpy(wl.k)
    mu, sg, _ = oracle_summaries(wl, kn, sub_block=sub)
    mlo, mhi, slo, shi = f16_record_ranges(wl, kn, mu, sg, sub_block=sub, rnd=oracle.round_e4m3)
    same = total = 0
    for bb in range(B):
        N = lens[bb] // b
        for name in ("mu", "sigma"):
            g8 = _f64(getattr(s8, name)[bb, ..., :N])
            g32 = _f64(getattr(s32, name)[bb, ..., :N])
            np.testing.assert_array_equal(g8, oracle.round_e4m3(g32), err_msg=name)
        assert torch.equal(s8.max_norm[bb, :, :N], s32.max_norm[bb, :, :N])
        for gpu, ref, lo, hi in ((s8.mu, mu, mlo, mhi), (s8.sigma, sg, slo, shi)):
            x = np.moveaxis(_f64(gpu[bb, :, :, :N]), -1, 1)
            r = oracle.round_e4m3(ref[bb, :, :N])
            assert np.all((x >= lo[bb, :, :N]) & (x <= hi[bb, :, :N]))
            same += int(np.sum(x == r))
            total += x.size
    say(f"[gpu] FP8 records equal to the oracle's rounding: {same}/{total}")
    assert same >= 0.995 * total


# fp32 values the statistics take exactly, with the E4M3 case each one exercises
MU_EDGES = [
    0.0, 1.0, -1.0,
    1.0625,          # tie between 1 and 1.125: to even (1)
    1.1875,          # tie between 1.125 and 1.25: to even (1.25)
    -1.0625,
    15.5,            # tie with a carry into the next binade (16)
    248.0,           # same at exponent 7 (256)
    240.0, 448.0,    # exact; largest finite
    456.0, 460.0,    # below the saturation tie: 448
    464.0, 470.0, 1000.0, -3000.0,   # saturated to +-448
    2.0 ** -6,       # smallest normal
    2.0 ** -9,       # smallest subnormal
    2.0 ** -10,      # tie between 0 and 2^-9: to even (0)
    3 * 2.0 ** -10,  # tie between 2^-9 and 2^-8: to even (2^-8)
    5 * 2.0 ** -10,  # tie between 2^-8 and 3 * 2^-9: to even (2^-8)
    -7 * 2.0 ** -10,
    0.0155029296875,  # just below 2^-6: the subnormal rounding reaches the smallest normal
    0.3125, 0.09375, -2.75, 37.0,
    0.0205078125,    # 21 * 2^-10: tie at the smallest normal exponent (to 10 * 2^-9)
]
SG_EDGES = [abs(x) for x in MU_EDGES if x != 0.0] + [0.0]


def test_fp8_encoder_edge_values():
    """Constant columns give mu = c exactly (sigma 0); columns alternating +-delta
    give mu 0 and sigma |delta| exactly (every value has at most 9 significant
    bits, so each fp32 partial sum of up to 64 terms, and of their squares, is
    exact); the FP8 codes must be the E4M3 rounding of those exact values."""
    B, Hkv, d, b = 1, 1, 64, 64
    nE, nS = len(MU_EDGES), len(SG_EDGES)
    N = 2 * max(nE, nS)
    T = N * b
    kk = np.zeros((B, Hkv, T, d), np.float32)
    want_mu = np.zeros((N, d))
    want_sg = np.zeros((N, d))
    sign = np.where(np.arange(b) % 2 == 0, 1.0, -1.0)
    for j in range(N):
        for i in range(d):
            if j % 2 == 0:
                c = np.float32(MU_EDGES[(i + j) % nE])
                kk[0, 0, j * b:(j + 1) * b, i] = c
                want_mu[j, i] = float(c)
            else:
                dl = np.float32(SG_EDGES[(i + 3 * j) % nS])
                kk[0, 0, j * b:(j + 1) * b, i] = dl * sign
                want_sg[j, i] = float(dl)
    dev = torch.device("cuda")
    k = torch.from_numpy(kk).to(dev)
    sl = torch.tensor([T], dtype=torch.int32, device=dev)
    s32 = eta.build_block_summaries(k, sl, b)
    s8 = eta.build_block_summaries(k, sl, b, stat_dtype=FP8)
    torch.cuda.synchronize()
    m32, g32 = _f64(s32.mu[0, 0]).T, _f64(s32.sigma[0, 0]).T     # [N][d]
    np.testing.assert_array_equal(m32, want_mu)
    np.testing.assert_array_equal(g32, want_sg)
    m8, g8 = _f64(s8.mu[0, 0]).T, _f64(s8.sigma[0, 0]).T
    np.testing.assert_array_equal(m8, oracle.round_e4m3(want_mu))
    np.testing.assert_array_equal(g8, oracle.round_e4m3(want_sg))
    # a few of the cases above, spelled out
    e = oracle.round_e4m3(np.array([1.0625, 1.1875, 15.5, 464.0, 1000.0, 2.0 ** -10, 3 * 2.0 ** -10]))
    assert list(e) == [1.0, 1.25, 16.0, 448.0, 448.0, 0.0, 2.0 ** -8]
    # the stored bytes are the OCP E4M3 codes torch decodes (largest finite: 0x7e)
    codes = s8.mu[0, 0].view(torch.uint8).cpu()
    assert int((codes & 0x7f).max()) == 0x7e


UPDATE_CASES = [
    # d, b, prev lens, new lens, max_new_blocks, sub_block
    (128, 64, [64 * 20 + 3, 64 * 5, 0], [64 * 23 + 1, 64 * 5 + 63, 64 * 2], 3, 0),
    (64, 128, [128 * 3 + 1], [128 * 9], 8, 4),
]


@pytest.mark.parametrize("case", range(len(UPDATE_CASES)))
def test_update_on_fp8_records_equals_full_build(case):
    d, b, prev, new, max_new, sub = UPDATE_CASES[case]
    B, Hkv = len(prev), 2
    T_cap = b * 32
    wl = make_workload(B=B, Hq=4, Hkv=Hkv, d=d, block=b, seq_lens=[T_cap] * B, T_cap=T_cap,
                       planted={"frac": 0.1}, predictor=False, tau_const=1.0, seed=150 + case)
    dev = torch.device("cuda")
    k = wl.k.to(dev)
    pl = torch.tensor(prev, dtype=torch.int32, device=dev)
    nl = torch.tensor(new, dtype=torch.int32, device=dev)
    full = eta.build_block_summaries(k, nl, b, sub_block=sub, stat_dtype=FP8)
    s = eta.build_block_summaries(k, pl, b, sub_block=sub, stat_dtype=FP8)
    eta.update_block_summaries(k, pl, nl, s, b, max_new_blocks=max_new, sub_block=sub)
    torch.cuda.synchronize()
    for bb in range(B):
        n_n = new[bb] // b
        for name in ("mu", "sigma"):
            x = getattr(s, name)[bb, ..., :n_n].view(torch.uint8)
            y = getattr(full, name)[bb, ..., :n_n].view(torch.uint8)
            assert torch.equal(x, y), (bb, name)
        assert torch.equal(s.max_norm[bb, :, :n_n], full.max_norm[bb, :, :n_n])


FP8_DECODE = {
    "gqa4_d128_b64": dict(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[20000, 9001],
                          planted={"frac": 0.05}, predictor=True, target_survival=0.15, seed=190),
    "gqa8_d64_b128": dict(B=1, Hq=16, Hkv=2, d=64, block=128, seq_lens=[40000],
                          planted={"frac": 0.03}, predictor=True, target_survival=0.2, seed=191),
    "gqa4_d128_b128_const": dict(B=1, Hq=8, Hkv=2, d=128, block=128, seq_lens=[30000],
                                 planted={"frac": 0.05}, predictor=False, tau_const=2.0, seed=192),
    # 16 screening tiles: the FP8 screening pairs neighbouring tiles on one XCD
    "gqa4_d128_b64_16tiles": dict(B=1, Hq=8, Hkv=2, d=128, block=64, seq_lens=[65536 - 37],
                                  planted={"frac": 0.03}, predictor=True, target_survival=0.2,
                                  seed=193),
}


@pytest.mark.parametrize("name", sorted(FP8_DECODE))
def test_decode_on_fp8_records_matches_oracle(name):
    wl = make_workload(**FP8_DECODE[name])
    np_in = oracle_inputs(wl)
    calibrate_bias(wl, np_in)
    g = run_gpu(wl, stat_dtype=FP8)
    mu, sg, mx = oracle_summaries(wl, np_in[1])
    mu8, sg8 = oracle.round_e4m3(mu), oracle.round_e4m3(sg)
    orc, tau_o = run_oracle(wl, np_in, summaries=(mu8, sg8, mx))
    extra = f16_band(wl, np_in[0], mu8, sg8,
                     f16_record_ranges(wl, np_in[1], mu, sg, rnd=oracle.round_e4m3))
    stats = compare(wl, g, orc, tau_o, np_inputs=np_in, band_extra=extra,
                    union_counts=g.union_counts)
    say(f"[gpu] FP8 index {name}: {stats}, median band {float(np.median(extra)):.2e}, "
        f"max band {float(np.max(extra)):.2e}")


def test_fp8_bounds_on_paired_tiles_match_the_oracle():
    """eta_block_bounds on FP8 records with 32 screening tiles (the paired tile
    order) against the oracle's bounds from its own E4M3-rounded records: fp32
    evaluation of the same bound, so within a few fp32 ulps of the bound's
    terms (plus the record intervals next to rounding midpoints)."""
    wl = make_workload(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[2048 * 64, 2048 * 64 - 5000],
                       planted={"frac": 0.03}, predictor=False, tau_const=1.0, seed=194)
    np_in = oracle_inputs(wl)
    dev = torch.device("cuda")
    k = wl.k.to(dev)
    sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
    s8 = eta.build_block_summaries(k, sl, wl.block, num_q_heads=wl.Hq, stat_dtype=FP8)
    gb = eta.block_bounds(wl.q.to(dev), sl, s8, k, block_size=wl.block, z=wl.z).cpu().numpy()
    mu, sg, mx = oracle_summaries(wl, np_in[1])
    mu8, sg8 = oracle.round_e4m3(mu), oracle.round_e4m3(sg)
    r = oracle.decode(np_in[0], np_in[1], np_in[2], wl.seq_lens, None, block_size=wl.block,
                      z=wl.z, bounds_only=True, summaries=(mu8, sg8, mx))
    extra = f16_band(wl, np_in[0], mu8, sg8,
                     f16_record_ranges(wl, np_in[1], mu, sg, rnd=oracle.round_e4m3))
    worst = 0.0
    for b in range(wl.B):
        N = wl.seq_lens[b] // wl.block
        ob, g = r.bounds[b, :, :N], gb[b, :, :N].astype(np.float64)
        err = np.abs(g - ob) - extra[b, :, :N]
        tol = 1e-5 * np.maximum(1.0, np.abs(ob))
        assert np.all(err <= tol), (b, float(np.max(err - tol)))
        worst = max(worst, float(np.max(np.abs(g - ob))))
    say(f"[gpu] FP8 bounds on 32 tiles: largest difference {worst:.2e}")

