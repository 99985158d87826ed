"""GPU parity of the half-precision block index (fp16 mu / sigma records, fp32 M;
App. "GQA-Grouped Execution and Compact Metadata Layout"); needs an MI355X.

  * the fp16 records are the fp32 statistics rounded to nearest even, bit for
    bit (self-consistency with the fp32 build); each lies in the interval of
    fp16 values that rounding any fp32 statistic within the summation error
    bound of the oracle's fp64 one can give (gpu_support.f16_record_ranges),
    which is the oracle's own rounding (oracle.round_f16) except next to a
    rounding midpoint; M is the fp32 build's;
  * a decode step screening on fp16 records matches the oracle screening on its
    own fp16-rounded records, with the tie band widened by the largest bound
    change those intervals allow (gpu_support.f16_band).
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


@pytest.fixture(autouse=True)
def _gpu(request):
    require_gpu()
    say(f"\n[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


F16_CASES = [
    # Hkv, d, b, lens, dtype, sub_block
    (2, 128, 128, [128 * 60 + 5], torch.bfloat16, 0),
    (2, 128, 64, [64 * 70, 64 * 3 + 1], torch.bfloat16, 0),
    (1, 64, 64, [64 * 40], torch.float32, 0),
    (2, 128, 64, [64 * 50 + 7], torch.bfloat16, 4),
]


@pytest.mark.parametrize("case", range(len(F16_CASES)))
def test_f16_records_are_rounded_statistics(case):
    Hkv, d, b, lens, dt, sub = F16_CASES[case]
    B = len(lens)
    wl = make_workload(B=B, Hq=Hkv, Hkv=Hkv, d=d, block=b, seq_lens=lens, dtype=dt,
                       planted={"frac": 0.1}, predictor=False, tau_const=1.0, seed=80 + case)
    dev = torch.device("cuda")
    k = wl.k.to(dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    s32 = eta.build_block_summaries(k, sl, b, sub_block=sub)
    s16 = eta.build_block_summaries(k, sl, b, sub_block=sub, stat_dtype=torch.float16)
    torch.cuda.synchronize()
    assert s16.mu.dtype == torch.float16 and s16.max_norm.dtype == torch.float32
    kn = as_numpy(wl.k)
    mu, sg, _ = oracle_summaries(wl, kn, sub_block=sub)
    mlo, mhi, slo, shi = f16_record_ranges(wl, kn, mu, sg, sub_block=sub)
    same = total = 0
    for bb in range(B):
        N = lens[bb] // b
        for name in ("mu", "sigma"):
            g16 = getattr(s16, name)[bb, ..., :N]
            g32 = getattr(s32, name)[bb, ..., :N]
            assert torch.equal(g16, g32.to(torch.float16)), name
        assert torch.equal(s16.max_norm[bb, :, :N], s32.max_norm[bb, :, :N])
        for gpu, ref, lo, hi in ((s16.mu, mu, mlo, mhi), (s16.sigma, sg, slo, shi)):
            x = np.moveaxis(gpu[bb, :, :, :N].float().cpu().numpy().astype(np.float64), -1, 1)
            r = oracle.round_f16(ref[bb, :, :N])
            assert np.all((x >= lo[bb, :, :N]) & (x <= hi[bb, :, :N]))
            same += int(np.sum(x == r))
            total += x.size
    say(f"[gpu] fp16 records equal to the oracle's rounding: {same}/{total}")
    assert same >= 0.99 * total


F16_DECODE = {
    "gqa4_d128_b64": dict(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[20000, 9001],
                          planted={"frac": 0.05}, predictor=True, target_survival=0.15, seed=90),
    "gqa8_d64_b128": dict(B=1, Hq=16, Hkv=2, d=64, block=128, seq_lens=[40000],
                          planted={"frac": 0.03}, predictor=True, target_survival=0.2, seed=91),
    "gqa4_d128_b128_const": dict(B=1, Hq=8, Hkv=2, d=128, block=128, seq_lens=[30000],
                                 planted={"frac": 0.05}, predictor=False, tau_const=2.0, seed=92),
}


@pytest.mark.parametrize("name", sorted(F16_DECODE))
def test_decode_on_f16_records_matches_oracle(name):
    wl = make_workload(**F16_DECODE[name])
    np_in = oracle_inputs(wl)
    calibrate_bias(wl, np_in)
    g = run_gpu(wl, stat_dtype=torch.float16)
    mu, sg, mx = oracle_summaries(wl, np_in[1])
    mu16, sg16 = oracle.round_f16(mu), oracle.round_f16(sg)
    orc, tau_o = run_oracle(wl, np_in, summaries=(mu16, sg16, mx))
    extra = f16_band(wl, np_in[0], mu16, sg16, f16_record_ranges(wl, np_in[1], mu, sg))
    stats = compare(wl, g, orc, tau_o, np_inputs=np_in, band_extra=extra,
                    union_counts=g.union_counts)
    say(f"[gpu] fp16 index {name}: {stats}, median band {float(np.median(extra)):.2e}")
