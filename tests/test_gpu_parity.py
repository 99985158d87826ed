"""GPU parity of the HIP path against the fp64 oracle (needs an MI355X).

Every test calls the C ABI through the binding on cuda:0 and compares with the
oracle on the same seeded inputs, element by element: at sizes that span several
screening tiles and a ragged tail, and on every (sequence, head) row of the full
workloads -- the 512K one through the benchmark's own prepared call at each
point of its survival sweep.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from gpu_support import (GpuRun, calibrate_bias, compare, f16_band, f16_record_ranges,
                         oracle_inputs, oracle_summaries, require_gpu, run_gpu, run_oracle, say)
from paper_2609_20888_amd import eta
from synth import as_numpy, config1, config2, config3, config4, config5, make_workload, place_bias

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(request):
    require_gpu()
    say(f"\n[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


# ------------------------------------------------------------------ building blocks

SUMMARY_CASES = [
    # B, Hkv, d, b, lens, dtype
    (2, 2, 128, 64, [20000, 17001], torch.bfloat16),
    (1, 3, 64, 128, [9000], torch.bfloat16),
    (2, 1, 64, 64, [5000, 63], torch.float32),
    (1, 2, 128, 128, [128 * 40 + 5], torch.float32),
    (1, 2, 128, 128, [128 * 70 + 17], torch.bfloat16),
    (2, 1, 64, 64, [64 * 33, 64 * 32], torch.bfloat16),
    (1, 1, 128, 64, [64 * 50 + 1], torch.float32),
    (1, 2, 64, 128, [128 * 31], torch.float32),
]


@pytest.mark.parametrize("case", range(len(SUMMARY_CASES)))
def test_block_summaries_match_oracle(case):
    B, Hkv, d, b, lens, dt = SUMMARY_CASES[case]
    wl = make_workload(B=B, Hq=Hkv, Hkv=Hkv, d=d, block=b, seq_lens=lens, dtype=dt,
                       planted={"frac": 0.1}, predictor=False, tau_const=1.0, seed=case)
    dev = torch.device("cuda")
    k = wl.k.to(dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    s = eta.build_block_summaries(k, sl, b)
    torch.cuda.synchronize()
    mu, sg, mx = s.mu.cpu().numpy(), s.sigma.cpu().numpy(), s.max_norm.cpu().numpy()
    kn = as_numpy(wl.k)
    for bb in range(B):
        for g in range(Hkv):
            N = lens[bb] // b
            omu, osg, omx = oracle.summaries(kn[bb, g, :lens[bb]], b)
            np.testing.assert_allclose(mu[bb, g, :, :N].T, omu, rtol=1e-5, atol=1e-5)
            np.testing.assert_allclose(sg[bb, g, :, :N].T, osg, rtol=1e-5, atol=1e-5)
            np.testing.assert_allclose(mx[bb, g, :N], omx, rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("Hq,d", [(16, 128), (32, 128), (4, 64), (12, 64),
                                  (6, 37), (5, 3), (1, 1024)])   # Hq d not a multiple of 4; Hq % 4 != 0
def test_predict_threshold_matches_oracle(dt, Hq, d):
    g = torch.Generator().manual_seed(Hq * d)
    q = torch.randn(5, Hq, d, generator=g).to(dt)
    W = torch.randn(Hq * d, Hq, generator=g) * 0.02
    bias = torch.randn(Hq, generator=g)
    dev = torch.device("cuda")
    tau = eta.predict_threshold(q.to(dev), W.t().contiguous().to(dev), bias.to(dev)).cpu().numpy()
    ref = oracle.predict(as_numpy(q), W.numpy(), bias.numpy())
    np.testing.assert_allclose(tau, ref, rtol=1e-5, atol=1e-5)
    tau0 = eta.predict_threshold(q.to(dev), None, bias.to(dev)).cpu().numpy()
    np.testing.assert_array_equal(tau0, np.tile(bias.numpy(), (5, 1)))


@pytest.mark.parametrize("G,d,b,dt", [(4, 128, 64, torch.bfloat16), (8, 64, 128, torch.bfloat16),
                                      (1, 64, 64, torch.float32), (2, 128, 128, torch.float32)])
def test_block_bounds_match_oracle(G, d, b, dt):
    wl = make_workload(B=2, Hq=2 * G, Hkv=2, d=d, block=b, seq_lens=[b * 300 + 7, b * 3],
                       dtype=dt, planted={"frac": 0.05}, predictor=False, tau_const=1.0, seed=G)
    dev = torch.device("cuda")
    k = wl.k.to(dev)
    sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
    s = eta.build_block_summaries(k, sl, b, num_q_heads=wl.Hq)
    for z in (0.0, 1.0, 2.0, 50.0):
        gb = eta.block_bounds(wl.q.to(dev), sl, s, k, block_size=b, z=z).cpu().numpy()
        q, kn, vn = oracle_inputs(wl)
        r = oracle.decode(q, kn, vn, wl.seq_lens, None, block_size=b, z=z, bounds_only=True)
        for bb in range(2):
            N = wl.seq_lens[bb] // b
            np.testing.assert_allclose(gb[bb, :, :N], r.bounds[bb, :, :N], rtol=2e-5, atol=2e-5)
            assert np.all(np.isnan(gb[bb, :, N:]))


# ------------------------------------------------------------------ decode parity

DECODE_CASES = {
    # name: (workload kwargs, run kwargs)
    "gqa4_bf16_two_tiles_ragged": (dict(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[20000, 17000],
                                        planted={"frac": 0.05}, predictor=True, target_survival=0.1,
                                        seed=11), {}),
    "gqa8_bf16_d64_b128": (dict(B=1, Hq=16, Hkv=2, d=64, block=128, seq_lens=[40000],
                                planted={"frac": 0.03}, predictor=True, target_survival=0.2,
                                seed=12), {}),
    "mha_fp32_planted": (dict(B=2, Hq=2, Hkv=2, d=64, block=64, seq_lens=[5000, 130],
                              dtype=torch.float32, planted={"count": 6}, per_head_planting=True,
                              predictor=False, tau_const=2.0, seed=13), {}),
    "gqa2_fp32_b128_d128": (dict(B=2, Hq=4, Hkv=2, d=128, block=128, seq_lens=[9000, 300],
                                 dtype=torch.float32, planted={"frac": 0.1}, predictor=True,
                                 target_survival=0.3, seed=14), {}),
    "rescue_only": (dict(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[30000, 3000],
                         predictor=False, tau_const=50.0, seed=15), {}),
    "rescue_window_small": (dict(B=1, Hq=4, Hkv=1, d=64, block=64, seq_lens=[4000],
                                 predictor=False, tau_const=50.0, rescue_window=5, seed=16), {}),
    "rescue_off": (dict(B=1, Hq=4, Hkv=1, d=64, block=64, seq_lens=[4096 + 10],
                        predictor=False, tau_const=50.0, rescue_window=0, seed=17), {}),
    "pins": (dict(B=1, Hq=8, Hkv=2, d=128, block=64, seq_lens=[10000], predictor=False,
                  tau_const=50.0, lwb=2, seed=18), {}),
    "self_ungated": (dict(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[6401, 6400],
                          planted={"frac": 0.05}, predictor=True, target_survival=0.1, seed=19),
                     dict(self_ungated=True)),
    "screen_all_dense_gated": (dict(B=1, Hq=8, Hkv=2, d=128, block=64, seq_lens=[7777],
                                    predictor=False, tau_const=0.5, seed=20),
                               dict(screen_all=True)),
    "tau_minus_inf_plain_softmax": (dict(B=1, Hq=4, Hkv=4, d=64, block=64, seq_lens=[3000],
                                         predictor=False, tau_const=-math.inf, seed=21), {}),
    "tail_only_and_empty": (dict(B=3, Hq=4, Hkv=2, d=128, block=128, seq_lens=[50, 0, 127],
                                 T_cap=256, predictor=False, tau_const=1.0, seed=22), {}),
    "slack_offset": (dict(B=1, Hq=8, Hkv=2, d=128, block=64, seq_lens=[12345],
                          planted={"frac": 0.05}, predictor=False, tau_const=2.2, a=0.3, seed=23),
                     {}),
    "splits_1": (dict(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[20000, 640],
                      planted={"frac": 0.05}, predictor=True, target_survival=0.15, seed=24),
                 dict(num_splits=1)),
    # one sequence, one split per kv head: the split workgroup writes the output,
    # counts and union counts itself (no combine); bf16 with a tail, and fp32 with
    # every head rescued
    "single_split_bf16_tail": (dict(B=1, Hq=8, Hkv=2, d=128, block=64, seq_lens=[20000],
                                    planted={"frac": 0.05}, predictor=True, target_survival=0.15,
                                    seed=26), dict(num_splits=1)),
    "single_split_fp32_rescue": (dict(B=1, Hq=4, Hkv=1, d=64, block=64, seq_lens=[4000],
                                      dtype=torch.float32, predictor=False, tau_const=50.0,
                                      seed=27), dict(num_splits=1)),
    "splits_1024": (dict(B=1, Hq=8, Hkv=2, d=128, block=64, seq_lens=[20000],
                         planted={"frac": 0.05}, predictor=True, target_survival=0.15, seed=25),
                    dict(num_splits=1024)),
}


@pytest.mark.parametrize("name", sorted(DECODE_CASES))
def test_decode_matches_oracle(name):
    wkw, rkw = DECODE_CASES[name]
    wl = make_workload(**wkw)
    np_in = oracle_inputs(wl)
    calibrate_bias(wl, np_in)
    g = run_gpu(wl, **rkw)
    okw = {k: v for k, v in rkw.items() if k in ("screen_all", "self_ungated")}
    orc, tau_o = run_oracle(wl, np_in, **okw)
    stats = compare(wl, g, orc, tau_o, np_inputs=np_in, union_counts=g.union_counts, **okw)
    say(f"[gpu] {name}: {stats}")


def test_decode_fp32_query_on_bf16_cache():
    # fp32 q with bf16 K/V: the scores use the hi + lo bf16 split of q
    wl = make_workload(B=1, Hq=8, Hkv=2, d=128, block=64, seq_lens=[9000],
                       planted={"frac": 0.05}, predictor=True, target_survival=0.1, seed=31)
    wl.q = torch.randn(wl.q.shape, generator=torch.Generator().manual_seed(5))
    wl.W = wl.W.float()
    np_in = oracle_inputs(wl)
    calibrate_bias(wl, np_in)
    g = run_gpu(wl)
    orc, tau_o = run_oracle(wl, np_in)
    say(compare(wl, g, orc, tau_o, np_inputs=np_in, union_counts=g.union_counts))


@pytest.mark.parametrize("G,d,b,dt", [(4, 128, 128, torch.bfloat16), (8, 64, 64, torch.bfloat16),
                                      (1, 64, 64, torch.float32), (2, 128, 64, torch.bfloat16)])
def test_decode_predicted_equals_predict_then_decode(G, d, b, dt):
    # the fused predictor uses the stand-alone predictor's summation order:
    # thresholds, masks and outputs must be bit-identical to the two-call path
    wl = make_workload(B=3, Hq=2 * G, Hkv=2, d=d, block=b, seq_lens=[b * 90 + 5, b * 33, 70],
                       dtype=dt, planted={"frac": 0.05}, predictor=True, target_survival=0.15,
                       seed=50 + G)
    np_in = oracle_inputs(wl)
    calibrate_bias(wl, np_in)
    dev = torch.device("cuda")
    q, k, v = wl.q.to(dev), wl.k.to(dev), wl.v.to(dev)
    sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
    summ = eta.build_block_summaries(k, sl, b, num_q_heads=wl.Hq)
    W, bias = wl.W_heads.to(dev), wl.bias.to(dev)
    p = eta.decode_params(beta=wl.beta, z=wl.z, rescue_window=wl.rescue_window)
    tau = eta.predict_threshold(q, W, bias)
    ref = eta.decode(q, k, v, sl, summ, tau, block_size=b, params=p)
    tau_out = torch.full_like(tau, float("nan"))
    fused = eta.decode_predicted(q, k, v, sl, summ, W, bias, block_size=b, params=p,
                                 tau_out=tau_out)
    torch.cuda.synchronize()
    assert torch.equal(tau_out, tau)
    assert torch.equal(fused.mask, ref.mask) and torch.equal(fused.counts, ref.counts)
    assert torch.equal(fused.out, ref.out)
    # and the fused path against the oracle
    assert torch.equal(fused.union_counts, ref.union_counts)
    g = GpuRun(out=fused.out, mask=fused.mask, counts=fused.counts, tau=tau_out, summ=summ,
               union_counts=fused.union_counts)
    orc, tau_o = run_oracle(wl, np_in)
    say(compare(wl, g, orc, tau_o, np_inputs=np_in, union_counts=fused.union_counts))
    # constant thresholds through the fused entry point (W = NULL)
    fused0 = eta.decode_predicted(q, k, v, sl, summ, None, bias, block_size=b, params=p,
                                  tau_out=tau_out)
    torch.cuda.synchronize()
    assert torch.equal(tau_out, bias.expand_as(tau_out))
    ref0 = eta.decode(q, k, v, sl, summ, bias.expand_as(tau).contiguous(), block_size=b, params=p)
    torch.cuda.synchronize()
    assert torch.equal(fused0.out, ref0.out) and torch.equal(fused0.mask, ref0.mask)


def _bf16_ulp(x: torch.Tensor) -> torch.Tensor:
    """Spacing of bf16 numbers at |x| (8 significant bits)."""
    e = torch.floor(torch.log2(x.abs().clamp_min(2.0 ** -126)))
    return torch.pow(2.0, e - 7)


def test_decode_is_deterministic_and_split_invariant():
    """Same inputs, same bits; other split counts change only the fp32 rounding of the
    merge (the two-stage reduction is exact in real arithmetic): bf16 outputs within
    one bf16 ulp per element, fp32 outputs (fp32 query) within 1e-5 of the row's
    largest element."""
    wl = make_workload(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[30000, 20000],
                       planted={"frac": 0.05}, predictor=False, tau_const=1.6, seed=41)
    a = run_gpu(wl)
    b = run_gpu(wl)
    assert torch.equal(a.out, b.out) and torch.equal(a.mask, b.mask)
    assert torch.equal(a.counts, b.counts) and torch.equal(a.union_counts, b.union_counts)
    worst_ulps = 0.0
    for s in (1, 5, 64, 300, 1024):
        r = run_gpu(wl, num_splits=s)
        assert torch.equal(r.mask, a.mask) and torch.equal(r.counts, a.counts)
        assert torch.equal(r.union_counts, a.union_counts)
        x, y = r.out.float(), a.out.float()
        ulps = ((x - y).abs() / _bf16_ulp(torch.maximum(x.abs(), y.abs()))).max().item()
        worst_ulps = max(worst_ulps, ulps)
        assert ulps <= 1.0, (s, ulps)
    wl.q = torch.randn(wl.q.shape, generator=torch.Generator().manual_seed(9))
    a32 = run_gpu(wl)
    worst32 = 0.0
    for s in (1, 5, 64, 300, 1024):
        r = run_gpu(wl, num_splits=s)
        assert torch.equal(r.mask, a32.mask)
        rel = ((r.out - a32.out).abs().amax(dim=-1) / a32.out.abs().amax(dim=-1)).max().item()
        worst32 = max(worst32, rel)
        assert rel <= 1e-5, (s, rel)
    say(f"[gpu] split invariance: bf16 worst {worst_ulps:.2f} ulp, fp32 worst {worst32:.2e} of row max")


def test_dense_decode_matches_oracle():
    for dt, d, b, lens in ((torch.bfloat16, 128, 64, [20000, 333]), (torch.float32, 64, 128, [5000])):
        wl = make_workload(B=len(lens), Hq=8, Hkv=2, d=d, block=b, seq_lens=lens, dtype=dt,
                           predictor=False, tau_const=0.0, seed=d)
        dev = torch.device("cuda")
        sl = torch.tensor(lens, dtype=torch.int32, device=dev)
        q, k, v = oracle_inputs(wl)
        r = oracle.decode(q, k, v, lens, np.zeros((wl.B, 8)), block_size=b, screen_all=True,
                          gate_off=True)
        tol = 2e-2 if dt == torch.bfloat16 else 1e-4
        # the library's split count, and one split per (sequence, kv head), where
        # the split workgroup writes the output and no combine runs
        for splits in (0, 1):
            out = eta.dense_decode(wl.q.to(dev), wl.k.to(dev), wl.v.to(dev), sl, block_size=b,
                                   num_splits=splits)
            torch.cuda.synchronize()
            o = out.float().cpu().numpy()
            for bb in range(wl.B):
                for h in range(8):
                    ref = r.o[bb, h]
                    assert np.max(np.abs(o[bb, h] - ref)) / np.max(np.abs(ref)) <= tol, (splits, bb, h)


# ------------------------------------------------------------------ full-size workloads

def test_config1_full():
    wl = config1()
    np_in = oracle_inputs(wl)
    g = run_gpu(wl)
    orc, tau_o = run_oracle(wl, np_in)
    stats = compare(wl, g, orc, tau_o, np_inputs=np_in, union_counts=g.union_counts)
    # every planted block and nothing else
    for h in range(4):
        assert np.nonzero(g.mask[0, h].cpu().numpy())[0].tolist() == wl.planted[(0, h)].tolist()
    say(stats)


def test_config2_full():
    wl = config2()
    np_in = oracle_inputs(wl)
    calibrate_bias(wl, np_in)
    g = run_gpu(wl)
    orc, tau_o = run_oracle(wl, np_in)
    say(compare(wl, g, orc, tau_o, np_inputs=np_in, union_counts=g.union_counts))


def _all_rows(wl):
    """Every (sequence, head) row of a full-size workload against the oracle (block
    index computed once by the oracle and shared by the bias placement and the decode)."""
    np_in = oracle_inputs(wl)
    osumm = oracle.block_index(np_in[1], wl.seq_lens, wl.block)
    calibrate_bias(wl, np_in, summaries=osumm)
    g = run_gpu(wl)
    orc, tau_o = run_oracle(wl, np_in, summaries=osumm)
    stats = compare(wl, g, orc, tau_o, np_inputs=np_in, union_counts=g.union_counts)
    assert stats["compared"] == wl.B * wl.Hq
    return stats


def test_config3_all_rows():
    say(_all_rows(config3(device="cuda")))


def test_config4_benchmarked_step_all_heads():
    """The benchmark's own call at the benchmark's shape: a prepared
    eta_decode_predicted step (predictor fused into screening, library-default
    splits) on the 512K workload, at the four survival points of the sweep, every
    query head against the oracle."""
    wl = config4(device="cuda")
    np_in = oracle_inputs(wl)
    q, k, v = np_in
    osumm = oracle.block_index(k, wl.seq_lens, wl.block)
    r0 = oracle.decode(q, k, v, wl.seq_lens, None, block_size=wl.block, z=wl.z, bounds_only=True,
                       summaries=osumm)
    W = as_numpy(wl.W)
    qW = oracle.predict(q, W, None)
    nb = [t // wl.block for t in wl.seq_lens]
    dev = torch.device("cuda")
    sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
    summ = eta.build_block_summaries(wl.k, sl, wl.block, num_q_heads=wl.Hq)
    bias_buf = torch.empty(wl.Hq, dtype=torch.float32, device=dev)
    params = eta.decode_params(beta=wl.beta, z=wl.z, offset_a=wl.a, rescue_window=wl.rescue_window)
    step = eta.DecodeStep(wl.q, wl.k, wl.v, sl, summ, wl.W_heads, bias_buf, block_size=wl.block,
                          params=params)
    for surv in (0.01, 0.05, 0.20, 1.0):
        bias = place_bias(r0.bounds, nb, qW, surv, wl.a)
        bias_buf.copy_(torch.as_tensor(bias, device=dev))
        step.run()
        torch.cuda.synchronize()
        wl.bias = torch.as_tensor(bias)
        tau_o = oracle.predict(q, W, bias)
        assert np.max(np.abs(step.tau.cpu().numpy() - tau_o)) <= 1e-5
        orc, _ = run_oracle(wl, np_in, tau=tau_o, summaries=osumm)
        g = GpuRun(out=step.out, mask=step.mask, counts=step.counts, tau=step.tau, summ=summ,
                   union_counts=step.union_counts)
        stats = compare(wl, g, orc, tau_o, np_inputs=np_in, union_counts=step.union_counts)
        assert stats["compared"] == wl.Hq and stats["union_counts_checked"] == wl.Hkv
        say(f"[gpu] 512K step at {surv:.0%} survival: {stats}")


@pytest.mark.parametrize("rec", ["f16", "fp8"])
def test_config4_benchmarked_step_compact_records(rec):
    """The benchmark's fp16 / FP8 record arms at the benchmark's shape: the
    prepared eta_decode_predicted step on the 512K workload's compact index at
    20% survival (thresholds placed from that index's own bounds, as the
    benchmark places them), every query head against the oracle screening the
    same rounded records, the tie band widened by the rounding intervals."""
    sd = torch.float16 if rec == "f16" else torch.float8_e4m3fn
    rnd = oracle.round_f16 if rec == "f16" else oracle.round_e4m3
    wl = config4(device="cuda")
    np_in = oracle_inputs(wl)
    q, k, v = np_in
    mu, sg, mx = oracle_summaries(wl, k)
    osumm = (rnd(mu), rnd(sg), mx)
    r0 = oracle.decode(q, k, v, wl.seq_lens, None, block_size=wl.block, z=wl.z, bounds_only=True,
                       summaries=osumm)
    W = as_numpy(wl.W)
    nb = [t // wl.block for t in wl.seq_lens]
    bias = place_bias(r0.bounds, nb, oracle.predict(q, W, None), 0.20, wl.a)
    dev = torch.device("cuda")
    sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
    summ = eta.build_block_summaries(wl.k, sl, wl.block, num_q_heads=wl.Hq, stat_dtype=sd)
    params = eta.decode_params(beta=wl.beta, z=wl.z, offset_a=wl.a, rescue_window=wl.rescue_window)
    bias_t = torch.as_tensor(bias, dtype=torch.float32, device=dev)
    step = eta.DecodeStep(wl.q, wl.k, wl.v, sl, summ, wl.W_heads, bias_t, block_size=wl.block,
                          params=params)
    step.run()
    torch.cuda.synchronize()
    wl.bias = torch.as_tensor(bias)
    tau_o = oracle.predict(q, W, bias)
    assert np.max(np.abs(step.tau.cpu().numpy() - tau_o)) <= 1e-5
    orc, _ = run_oracle(wl, np_in, tau=tau_o, summaries=osumm)
    extra = f16_band(wl, q, osumm[0], osumm[1], f16_record_ranges(wl, k, mu, sg, rnd=rnd))
    g = GpuRun(out=step.out, mask=step.mask, counts=step.counts, tau=step.tau, summ=summ,
               union_counts=step.union_counts)
    stats = compare(wl, g, orc, tau_o, np_inputs=np_in, band_extra=extra,
                    union_counts=step.union_counts)
    assert stats["compared"] == wl.Hq and stats["union_counts_checked"] == wl.Hkv
    say(f"[gpu] 512K step on {rec} records at 20% survival: {stats}")


def test_config5_constant_thresholds_all_rows():
    say(_all_rows(config5(device="cuda")))


def test_config5_predictor_all_rows():
    say(_all_rows(config5(device="cuda", predictor=True)))


def test_decode_predicted_predicts_once_per_step_past_the_fused_limit():
    """At the 32-sequence ragged shape (32/8 heads, 64K capacity) the screening
    workgroups would re-read ~268 MB of W per step, so eta_decode_predicted runs
    the stand-alone predictor first: one predict launch, and thresholds, mask,
    counts and output bit-identical to eta_predict_threshold + eta_decode; a
    small batch keeps the predictor fused (no predict launch)."""
    dev = torch.device("cuda")
    for wl, launches in ((config5(device="cuda", predictor=True), 1),
                         (make_workload(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[9000, 4000],
                                        planted={"frac": 0.05}, predictor=True,
                                        target_survival=0.2, seed=61), 0)):
        if launches == 0:
            calibrate_bias(wl)
        q, k, v = wl.q.to(dev), wl.k.to(dev), wl.v.to(dev)
        sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
        summ = eta.build_block_summaries(k, sl, wl.block, num_q_heads=wl.Hq)
        W, bias = wl.W_heads.to(dev), wl.bias.to(dev)
        p = eta.decode_params(beta=wl.beta, z=wl.z, rescue_window=wl.rescue_window)
        tau = eta.predict_threshold(q, W, bias)
        ref = eta.decode(q, k, v, sl, summ, tau, block_size=wl.block, params=p)
        tau_out = torch.full_like(tau, float("nan"))
        torch.cuda.synchronize()
        eta.profile_begin()
        fused = eta.decode_predicted(q, k, v, sl, summ, W, bias, block_size=wl.block, params=p,
                                     tau_out=tau_out)
        torch.cuda.synchronize()
        kt = eta.profile_end()
        assert kt["predict"][1] == launches, (wl.name, kt)
        assert torch.equal(tau_out, tau)
        assert torch.equal(fused.mask, ref.mask) and torch.equal(fused.counts, ref.counts)
        assert torch.equal(fused.out, ref.out)
        say(f"[gpu] {wl.name}: predict launches {launches}, union "
            f"{float(fused.mask.float().mean()):.3f}")
        del q, k, v, summ, ref, fused, wl
        torch.cuda.empty_cache()



@pytest.mark.parametrize("predictor", [True, False])
def test_decode_step_replays_in_a_hip_graph_like_eager(predictor):
    """A prepared decode step captured in a HIP graph (the serving loop's form):
    replayed four times, with eager work and synchronisations between the
    replays, every replay reproduces the eager step bit for bit (output, mask,
    counts, thresholds).  The path records no memset nodes."""
    wl = make_workload(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[20000, 9001],
                       planted={"frac": 0.05}, predictor=predictor, target_survival=0.15,
                       tau_const=1.6, seed=71)
    if predictor:
        calibrate_bias(wl)
    dev = torch.device("cuda")
    q, k, v = wl.q.to(dev), wl.k.to(dev), wl.v.to(dev)
    sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
    summ = eta.build_block_summaries(k, sl, wl.block, num_q_heads=wl.Hq)
    W = wl.W_heads.to(dev) if wl.W is not None else None
    bias = wl.bias.to(dev)
    p = eta.decode_params(beta=wl.beta, z=wl.z, rescue_window=wl.rescue_window)
    eager = eta.DecodeStep(q, k, v, sl, summ, W, bias, block_size=wl.block, params=p)
    eager.run()
    torch.cuda.synchronize()
    ref = (eager.out.clone(), eager.mask.clone(), eager.counts.clone(), eager.tau.clone())
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        warm = eta.DecodeStep(q, k, v, sl, summ, W, bias, block_size=wl.block, params=p)
        warm.run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step = eta.DecodeStep(q, k, v, sl, summ, W, bias, block_size=wl.block, params=p)
        step.run()
    for r in range(4):
        step.out.zero_()
        step.mask.fill_(7)
        step.counts.fill_(-1)
        eager.run()                     # eager work on the same inputs between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = (step.out, step.mask, step.counts, step.tau)
        for name, x, y in zip(("out", "mask", "counts", "tau"), got, ref):
            assert torch.equal(x, y), (r, name)
    say(f"[gpu] graph replays of the decode step match eager (predictor={predictor})")


# ------------------------------------------------------------------ seeded random geometries

def _random_geometry(seed: int):
    """One seeded small geometry: group size, head dim, block size, K/V type, ragged
    lengths (some below one block, some with a tail), predictor or constant
    thresholds, rescue window, pinned blocks, split count."""
    rng = np.random.default_rng(1000 + seed)
    G = int(rng.choice([1, 2, 4, 8]))
    Hkv = int(rng.choice([1, 2])) if G < 8 else 1
    d = int(rng.choice([64, 128]))
    block = int(rng.choice([64, 128]))
    B = int(rng.integers(1, 4))
    lens = [int(rng.integers(0, 40 * block)) for _ in range(B)]
    if rng.random() < 0.3:
        lens[0] = int(rng.integers(0, block))               # shorter than one block
    dtype = torch.float32 if rng.random() < 0.25 else torch.bfloat16
    predictor = bool(rng.random() < 0.6)
    wkw = dict(B=B, Hq=G * Hkv, Hkv=Hkv, d=d, block=block, seq_lens=lens, dtype=dtype,
               planted={"frac": 0.05}, predictor=predictor, seed=2000 + seed,
               rescue_window=int(rng.choice([0, 3, 64, 256])), lwb=int(rng.choice([0, 0, 2])))
    if predictor:
        wkw["target_survival"] = float(rng.choice([0.02, 0.1, 0.3]))
    else:
        wkw["tau_const"] = float(rng.choice([0.5, 1.5, 3.0]))
    rkw = dict(num_splits=int(rng.choice([0, 0, 1, 3, 17])))
    return wkw, rkw


# The proportional plan with more (sequence, kv head) groups than a split
# workgroup has threads: thread t then takes groups t, t + 256, ... (all four
# rounds at 1024 groups, the most the plan takes), and with 3 kv heads the
# groups' sequence indexes step with carries.  One 64-block screening tile per
# group keeps every tile count in the plan's table.
MANY_GROUPS = {
    "320_groups_predictor": dict(B=160, Hq=4, Hkv=2, d=64, block=64, T_cap=4096, predictor=True,
                                 target_survival=0.1),
    "300_groups_3_kv_heads": dict(B=100, Hq=6, Hkv=3, d=64, block=64, T_cap=2048, predictor=False,
                                  tau_const=1.5),
    "1024_groups_predictor": dict(B=512, Hq=4, Hkv=2, d=64, block=64, T_cap=1024, predictor=True,
                                  target_survival=0.1),
}


@pytest.mark.parametrize("name", sorted(MANY_GROUPS))
def test_proportional_plan_many_groups(name):
    kw = dict(MANY_GROUPS[name])
    rng = np.random.default_rng(len(name))
    lens = rng.integers(0, kw["T_cap"] + 1, size=kw["B"]).tolist()
    groups, tiles = kw["B"] * kw["Hkv"], (kw["T_cap"] // kw["block"] + 63) // 64
    assert 256 < groups <= 1024 and groups * tiles <= 4096      # the proportional plan's table
    wl = make_workload(**kw, seq_lens=lens, planted={"frac": 0.05}, seed=4000 + len(name))
    np_in = oracle_inputs(wl)
    calibrate_bias(wl, np_in)
    g = run_gpu(wl)
    orc, tau_o = run_oracle(wl, np_in)
    stats = compare(wl, g, orc, tau_o, np_inputs=np_in, union_counts=g.union_counts)
    say(f"[gpu] {name}: {stats}")
    assert stats["compared"] == wl.B * wl.Hq


@pytest.mark.parametrize("num_splits", [0, 3])
def test_uniform_plan_many_sequences(num_splits):
    # More (sequence, kv head) groups than the proportional plan's table holds
    # (1040 > 1024): the uniform plan on a (S, Hkv, B) grid with B = 520, by
    # default one split per group (the split workgroup writes the output, no
    # combine), else three splits per group and the combine.
    rng = np.random.default_rng(77)
    lens = rng.integers(0, 1025, size=520).tolist()
    wl = make_workload(B=520, Hq=4, Hkv=2, d=64, block=64, seq_lens=lens, T_cap=1024,
                       planted={"frac": 0.05}, predictor=True, target_survival=0.2, seed=78)
    np_in = oracle_inputs(wl)
    calibrate_bias(wl, np_in)
    g = run_gpu(wl, num_splits=num_splits)
    orc, tau_o = run_oracle(wl, np_in)
    stats = compare(wl, g, orc, tau_o, np_inputs=np_in, union_counts=g.union_counts)
    say(f"[gpu] uniform plan, 520 sequences, splits {num_splits}: {stats}")
    assert stats["compared"] == wl.B * wl.Hq


@pytest.mark.parametrize("seed", range(12))
def test_decode_random_geometries(seed):
    wkw, rkw = _random_geometry(seed)
    say(f"[gpu] random geometry {seed}: {wkw} {rkw}")
    wl = make_workload(**wkw)
    np_in = oracle_inputs(wl)
    calibrate_bias(wl, np_in)
    g = run_gpu(wl, **rkw)
    orc, tau_o = run_oracle(wl, np_in)
    stats = compare(wl, g, orc, tau_o, np_inputs=np_in, union_counts=g.union_counts)
    assert stats["compared"] == wl.B * wl.Hq
