#!/usr/bin/env python3
"""Benchmark of the ETA decode step on one MI355X.

Workload: one decode step at 512K context -- batch 1, 16 query / 4 KV heads
(GQA 4), head_dim 128, KV blocks of 128 tokens, bf16 K/V ~N(0,1) with 1% of the
blocks planted query-aligned, thresholds from the linear predictor with the
bias placed for a given fraction of surviving blocks per head (synthetic data,
see the design doc).  A timed step is one eta_decode_predicted call (threshold
prediction fused into the screening launch, gated split decode over the
surviving blocks, combine, mask and counts); the KV cache and its block
summaries are resident in HBM before timing starts.  The summary
build (once per prefill) is timed on its own.

One JSON line on stdout:
  value           microseconds per decode step at 20% head survival, cold: the
                  mean GPU time of a step after a 512 MiB read sweep that flushes
                  the last-level cache (the back-to-back warm step beside it)
  roofline        achieved HBM bandwidth of the split-decode kernel (the
                  dominant one) on its algorithmic bytes; its average launch
                  duration comes from HIP events the library records on the
                  launch stream around each launch, in a pass of the same K
                  steps run right after the timed loop (the events are kept
                  out of the timed loop itself)
  cpu_baseline    the fp64 oracle timed on this host's cores on the same step
  sweep           the same step at 1% / 5% / 20% / 100% survival, cold and warm,
                  with the dense decode baseline at the same shape; the dense gated
                  (screen_all) arm; compact fp16 / FP8 records
  other_configs   4K MHA fp32, 32K GQA, 8 x 128K GQA and the 32 ragged sequences
                  (constants and predictor), each cold and warm with its dense
                  decode baseline
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PRIMARY_SURVIVAL = 0.20
SWEEP = (0.01, 0.05, 0.20, 1.00)
# sources of the decode-path kernels: the counter file's traffic is valid only for these
DECODE_SRCS = [os.path.join(ROOT, "paper_2609_20888_amd", "csrc", f)
               for f in ("eta_kernels.hip", "eta_device.h", "eta_index.h", "eta_internal.h")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "split_decode_512k_traffic.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_src_sha() -> str:
    """Hash of the decode kernels' code (comments and whitespace removed, so a
    comment edit does not orphan the committed counter summary)."""
    h = hashlib.sha256()
    for path in DECODE_SRCS:
        with open(path, encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU time budget of the oracle baseline")
    ap.add_argument("--no-prefill", action="store_true",
                    help="skip the gated prefill forward measurement")
    ap.add_argument("--prefill-only", action="store_true",
                    help="measure only the gated prefill forward and print its JSON (profiling)")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the 8 x 128K and 32-sequence ragged decode timings")
    ap.add_argument("--no-calibration", action="store_true",
                    help="skip the offline threshold calibration measurement")
    ap.add_argument("--only-config", default=None,
                    choices=["4k", "32k", "128k", "ragged", "ragged_pred"],
                    help="measure only this other workload and print its JSON (profiling)")
    ap.add_argument("--only-primary", action="store_true",
                    help="time only the 20%% survival point (profiling runs)")
    ap.add_argument("--splits", type=int, default=0,
                    help="splits per (sequence, kv head); 0 = the library's default")
    ap.add_argument("--graph", action="store_true",
                    help="replay the step from a captured HIP graph")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run a plain device copy of this size (counter calibration)")
    return ap.parse_args()


def measure_prefill(torch, eta, dev):
    """Gated prefill / training forward: one 16K-token sequence at the ragged
    workload's head shape (32 query / 8 kv heads, d = 128), bf16, causal."""
    pB, pHq, pHkv, pT, pd = 1, 32, 8, 16384, 128
    g = torch.Generator(device=dev).manual_seed(10)
    pq = torch.randn(pB, pHq, pT, pd, generator=g, device=dev).to(torch.bfloat16)
    pk = torch.randn(pB, pHkv, pT, pd, generator=g, device=dev).to(torch.bfloat16)
    pv = torch.randn(pB, pHkv, pT, pd, generator=g, device=dev).to(torch.bfloat16)
    ptau = 0.5 + 0.5 * torch.randn(pB, pHq, pT, generator=g, device=dev)
    psl = torch.full((pB,), pT, dtype=torch.int32, device=dev)
    pout, pR, pL = eta.gated_prefill(pq, pk, pv, ptau, psl, beta=4.0)
    torch.cuda.synchronize()
    pms = batch_median_ms(torch, lambda: eta.gated_prefill(pq, pk, pv, ptau, psl, beta=4.0, out=pout,
                                                           R=pR, L=pL), reps=5)
    pflops = 4.0 * pd * pHq * pT * (pT + 1) / 2      # QK^T and p.V over the causal pairs
    prefill = {"workload": f"B={pB}, {pT} tokens, {pHq}/{pHkv} heads, d={pd}, bf16, causal",
               "ms": round(pms, 3), "tflops": round(pflops / pms / 1e9, 1),
               "frac_of_bf16_mfma_peak": round(pflops / pms / 1e9 / 2500.0, 4)}
    log(f"[bench] gated prefill: {prefill}")
    return prefill


def flush_buffer(torch, dev):
    """512 MiB (twice the 256 MB last-level cache) read by a sum before each cold step;
    a read sweep leaves no dirty lines whose write-back would overlap the step."""
    return torch.ones(512 << 18, dtype=torch.int32, device=dev)


def time_cold(torch, run, steps, flush):
    """Per-step GPU time (events on the launch stream around each step), each step
    after a last-level-cache flush; the flushes are outside the intervals.  Returns
    (mean, p10, p50, p90) in microseconds."""
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    for a, b in evs:
        flush.sum(dtype=torch.int64)
        a.record()
        run()
        b.record()
    torch.cuda.synchronize()
    d = sorted(a.elapsed_time(b) * 1e3 for a, b in evs)
    pick = lambda f: round(d[min(len(d) - 1, int(f * len(d)))], 2)
    return round(sum(d) / len(d), 2), pick(0.1), pick(0.5), pick(0.9)


def batch_median_ms(torch, fn, reps=10, batches=3):
    """Milliseconds per call: events around `reps` back-to-back calls, the median of
    `batches` such batches (after one untimed call)."""
    fn()
    out = []
    for _ in range(batches):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        out.append(a.elapsed_time(b) / reps)
    return sorted(out)[len(out) // 2]


def time_warm(torch, run, steps, warmup=5):
    """Back-to-back steps: wall clock between synchronisations, microseconds per step."""
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        run()
    torch.cuda.synchronize()
    return round((time.perf_counter() - t0) * 1e6 / steps, 2)


def step_bytes(wl, union_blocks, predictor: bool, stat_bytes: int = 4):
    """Algorithmic bytes of one decode step: the block records of every full block,
    the union's K and V blocks and the tails, q in and the output out, thresholds, the
    mask, and the predictor's W and bias when thresholds are predicted."""
    e = 4 if str(wl.dtype).endswith("float32") else 2
    nblk = [t // wl.block for t in wl.seq_lens]
    rec = 2 * wl.d * stat_bytes + 4
    tail = sum(t - n * wl.block for t, n in zip(wl.seq_lens, nblk)) * wl.Hkv
    kv = (union_blocks * wl.block + tail) * wl.d * e * 2
    records = sum(nblk) * wl.Hkv * rec
    small = wl.B * wl.Hq * wl.d * e * 2 + wl.B * wl.Hq * wl.n_blk_cap + wl.B * wl.Hq * 4 * 2
    if predictor:
        small += wl.Hq * wl.d * wl.Hq * 4 + wl.Hq * 4
    return kv, kv + records + small


def measure_compact(torch, np, eta, dev, wl, steps, flush, stat_dtype):
    """The same workload screened on half-precision (or FP8) records: thresholds
    placed from that index's own bounds (the same head survival), cold and warm
    step and per-kernel times."""
    from synth import place_bias
    sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
    summ = eta.build_block_summaries(wl.k, sl, wl.block, num_q_heads=wl.Hq, stat_dtype=stat_dtype)
    nblk = [t // wl.block for t in wl.seq_lens]
    W_h = wl.W_heads                    # head-major, as the library takes it
    if wl.W is not None:
        bounds = eta.block_bounds(wl.q, sl, summ, wl.k, block_size=wl.block, z=wl.z).cpu().numpy()
        qW = eta.predict_threshold(wl.q, W_h, torch.zeros(wl.Hq, device=dev)).cpu().numpy()
        bias = torch.as_tensor(place_bias(bounds, nblk, qW.astype(np.float64), wl.target_survival,
                                          wl.a), device=dev)
    else:
        bias = wl.bias.to(dev)
    p = eta.decode_params(beta=wl.beta, z=wl.z, offset_a=wl.a, rescue_window=wl.rescue_window,
                          lwb=wl.lwb)
    st = eta.DecodeStep(wl.q, wl.k, wl.v, sl, summ, W_h, bias, block_size=wl.block, params=p)
    warm = time_warm(torch, st.run, steps, warmup=10)
    cold = time_cold(torch, st.run, max(10, steps // 2), flush)[0]
    torch.cuda.synchronize()
    eta.profile_begin()
    for _ in range(20):
        st.run()
    torch.cuda.synchronize()
    kt = {name: round(t / n * 1e3, 2) for name, (t, n) in eta.profile_end().items() if n}
    return {"us_per_step_cold": cold, "us_per_step_warm": warm,
            "union_blocks": int(st.union_counts.sum()), "kernel_avg_us_warm": kt}


def measure_config(torch, np, eta, dev, wl, steps, flush, compact=False):
    """One workload at the library defaults: the prepared decode step (predicted or
    constant thresholds, the predictor bias placed from the GPU's own bounds) warm
    and cold, its union and algorithmic bytes, and the dense decode baseline at the
    same shape (cold and warm); with `compact`, also the step on fp16 records."""
    from synth import place_bias
    sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
    summ = eta.build_block_summaries(wl.k, sl, wl.block, num_q_heads=wl.Hq)
    nblk = [t // wl.block for t in wl.seq_lens]
    W_h = wl.W_heads                    # head-major, as the library takes it
    if wl.W is not None:
        bounds = eta.block_bounds(wl.q, sl, summ, wl.k, block_size=wl.block, z=wl.z).cpu().numpy()
        qW = eta.predict_threshold(wl.q, W_h, torch.zeros(wl.Hq, device=dev)).cpu().numpy()
        bias = torch.as_tensor(place_bias(bounds, nblk, qW.astype(np.float64), wl.target_survival,
                                          wl.a), device=dev)
    else:
        bias = wl.bias.to(dev)
    p = eta.decode_params(beta=wl.beta, z=wl.z, offset_a=wl.a, rescue_window=wl.rescue_window,
                          lwb=wl.lwb)
    st = eta.DecodeStep(wl.q, wl.k, wl.v, sl, summ, W_h, bias, block_size=wl.block, params=p)
    warm = time_warm(torch, st.run, steps, warmup=10)
    cold, c10, c50, c90 = time_cold(torch, st.run, max(10, steps // 2), flush)
    union = int(st.union_counts.sum())
    kv, total = step_bytes(wl, union, wl.W is not None)
    d_head = float(st.mask.float().sum()) / float(wl.Hq * sum(nblk))
    torch.cuda.synchronize()
    eta.profile_begin()
    for _ in range(20):
        st.run()
    torch.cuda.synchronize()
    kt = {name: round(t / n * 1e3, 2) for name, (t, n) in eta.profile_end().items() if n}
    dws = eta.alloc_workspace(eta.dense_workspace_size(eta.kv_desc(wl.k, wl.Hq, wl.block)), dev)
    dout = torch.empty_like(wl.q)
    dense = lambda: eta.dense_decode(wl.q, wl.k, wl.v, sl, block_size=wl.block, out=dout,
                                     workspace=dws)
    dense_warm = time_warm(torch, dense, max(10, steps // 2))
    dense_cold = time_cold(torch, dense, 10, flush)[0]
    r = {"us_per_step_cold": cold, "cold_p10_p50_p90": [c10, c50, c90], "us_per_step_warm": warm,
         "d_head": round(d_head, 4), "union_blocks": union,
         "d_union": round(union / float(wl.Hkv * sum(nblk)), 4),
         "step_bytes": total, "effective_GBps_cold": round(total / cold / 1e3, 1),
         "effective_frac_of_peak_cold": round(total / cold / 1e3 / HBM_PEAK_GBS, 4),
         "effective_GBps_warm": round(total / warm / 1e3, 1),
         "union_kv_GBps_cold": round(kv / cold / 1e3, 1),
         "dense_us_per_step_cold": dense_cold, "dense_us_per_step_warm": dense_warm,
         "speedup_vs_dense_cold": round(dense_cold / cold, 3),
         "speedup_vs_dense_warm": round(dense_warm / warm, 3), "kernel_avg_us_warm": kt}
    if compact:
        del st, summ
        torch.cuda.empty_cache()
        r["fp16_records"] = measure_compact(torch, np, eta, dev, wl, steps, flush, torch.float16)
    log(f"[bench] {wl.name}: {r}")
    return r


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the ETA decode path here is single-GPU; see DESIGN.md for how it would shard)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_20888_amd import eta
    from synth import config4, place_bias

    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    eta.load_library()
    if args.prefill_only:
        print(json.dumps({"gated_prefill": measure_prefill(torch, eta, dev)}), flush=True)
        return
    if args.only_config:
        from synth import config1, config2, config3, config5
        mk = {"4k": lambda: config1(device=dev), "32k": lambda: config2(device=dev),
              "128k": lambda: config3(device=dev), "ragged": lambda: config5(device=dev),
              "ragged_pred": lambda: config5(device=dev, predictor=True)}[args.only_config]
        r = measure_config(torch, np, eta, dev, mk(), args.steps, flush_buffer(torch, dev),
                           compact=args.only_config in ("128k", "ragged_pred"))
        print(json.dumps({args.only_config: r}), flush=True)
        return

    log("[bench] generating the 512K workload on the GPU")
    wl = config4(device=dev, survival=PRIMARY_SURVIVAL)
    B, Hq, Hkv, d, bs = wl.B, wl.Hq, wl.Hkv, wl.d, wl.block
    sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
    q, k, v, W = wl.q, wl.k, wl.v, wl.W_heads   # W head-major, as the library takes it
    e = 2  # bf16 bytes
    Ncap = wl.n_blk_cap
    torch.cuda.synchronize()

    # ---- summary build (prefill-time), timed on its own
    summ = eta.build_block_summaries(k, sl, bs, num_q_heads=Hq)
    torch.cuda.synchronize()
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    sum_ms = batch_median_ms(torch, lambda: eta.build_block_summaries(k, sl, bs, num_q_heads=Hq, out=summ))
    sum_bytes = B * Hkv * wl.seq_lens[0] * d * e + B * Hkv * (wl.seq_lens[0] // bs) * (2 * d * 4 + 4)
    log(f"[bench] summary build {sum_ms * 1e3:.1f} us ({sum_bytes / sum_ms / 1e6:.0f} GB/s)")

    # ---- index variants: sub-block envelope build (16 sub-blocks per block, as the
    # paper's b = 64 / b_sub = 4 layout) and the decode-time update when an appended
    # token completes a block in every (sequence, kv head)
    env_sub = bs // 16
    env = eta.build_block_summaries(k, sl, bs, num_q_heads=Hq, sub_block=env_sub)
    torch.cuda.synchronize()
    env_ms = batch_median_ms(torch, lambda: eta.build_block_summaries(k, sl, bs, num_q_heads=Hq,
                                                                      sub_block=env_sub, out=env))
    prev = sl - 1
    upd_reps = 50
    s0.record()
    for _ in range(upd_reps):
        eta.update_block_summaries(k, prev, sl, env, bs, max_new_blocks=1, num_q_heads=Hq)
    s1.record()
    torch.cuda.synchronize()
    upd_ms = s0.elapsed_time(s1) / upd_reps
    del env
    log(f"[bench] envelope build {env_ms * 1e3:.1f} us, per-step update {upd_ms * 1e3:.2f} us")

    # ---- thresholds: place the predictor bias from the GPU's own bounds
    bounds = eta.block_bounds(q, sl, summ, k, block_size=bs, z=wl.z).cpu().numpy()
    qW = eta.predict_threshold(q, W, torch.zeros(Hq, device=dev)).cpu().numpy().astype(np.float64)
    nblk = [t // bs for t in wl.seq_lens]
    biases = {s: torch.as_tensor(place_bias(bounds, nblk, qW, s, wl.a), device=dev) for s in SWEEP}

    params = eta.decode_params(beta=wl.beta, z=wl.z, offset_a=wl.a, rescue_window=wl.rescue_window,
                               num_splits=args.splits)
    desc = eta.kv_desc(k, Hq, bs)
    bias_buf = torch.empty(Hq, dtype=torch.float32, device=dev)
    # one prepared call per step: thresholds predicted inside the screening launch,
    # then the gated split decode over the surviving blocks and the combine
    prepared = eta.DecodeStep(q, k, v, sl, summ, W, bias_buf, block_size=bs, params=params)
    eager = prepared
    flush = flush_buffer(torch, dev)

    def set_point(bias):
        bias_buf.copy_(bias)
        torch.cuda.synchronize()

    graph = None
    if args.graph:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            prepared_g = eta.DecodeStep(q, k, v, sl, summ, W, bias_buf, block_size=bs,
                                        params=params, stream=side)
            for _ in range(3):
                prepared_g.run()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            prepared_c = eta.DecodeStep(q, k, v, sl, summ, W, bias_buf, block_size=bs,
                                        params=params)
            prepared_c.run()
        prepared = prepared_c

    def step():
        if graph is not None:
            graph.replay()
        else:
            prepared.run()

    def warm_percentiles(steps):
        """p10 / p50 / p90 of back-to-back single-step GPU times: one event between
        every two steps (each interval includes one event record, ~1-2 us)."""
        for _ in range(5):
            step()
        torch.cuda.synchronize()
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        evs[0].record()
        for i in range(steps):
            step()
            evs[i + 1].record()
        torch.cuda.synchronize()
        d = sorted(evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(steps))
        pick = lambda f: round(d[min(len(d) - 1, int(f * len(d)))], 2)
        return [pick(0.1), pick(0.5), pick(0.9)]

    def kernel_times(steps):
        """Per-kernel durations: HIP events recorded by the library around each launch."""
        torch.cuda.synchronize()
        eta.profile_begin()
        for _ in range(steps):
            eager.run()
        torch.cuda.synchronize()
        return eta.profile_end()

    # ---- dense decode at the same shape (plain softmax over every token)
    dws = eta.alloc_workspace(eta.dense_workspace_size(desc, args.splits), dev)
    dout = torch.empty_like(q)
    dense = lambda: eta.dense_decode(q, k, v, sl, block_size=bs, num_splits=args.splits,
                                     out=dout, workspace=dws)
    dense_warm = time_warm(torch, dense, max(10, args.steps // 4), warmup=3)
    dense_cold = time_cold(torch, dense, 20, flush)[0]
    dense_bytes = B * Hkv * wl.seq_lens[0] * d * e * 2
    log(f"[bench] dense decode cold {dense_cold:.1f} us, warm {dense_warm:.1f} us "
        f"({dense_bytes / dense_cold / 1e3:.0f} GB/s cold)")

    # ---- the survival sweep: cold steps (the headline at 20%) and back-to-back steps
    sweep = {}
    primary = None
    for s in (SWEEP if not args.only_primary else (PRIMARY_SURVIVAL,)):
        is_primary = abs(s - PRIMARY_SURVIVAL) < 1e-9
        set_point(biases[s])
        n_cold = args.steps if is_primary else max(20, args.steps // 4)
        warm = time_warm(torch, step, args.steps if is_primary else max(20, args.steps // 4),
                         warmup=args.warmup if is_primary else 5)
        cold, c10, c50, c90 = time_cold(torch, step, n_cold, flush)
        ub = int(prepared.union_counts.sum())
        kv_b, step_b = step_bytes(wl, ub, predictor=True)
        dh = float(prepared.mask[:, :, :nblk[0]].float().mean())
        du = ub / float(B * Hkv * nblk[0])
        entry = {"survival_target": s, "us_per_step_cold": cold, "cold_p10_p50_p90": [c10, c50, c90],
                 "us_per_step_warm": warm, "d_head": round(dh, 4), "d_union": round(du, 4),
                 "union_blocks": ub, "step_bytes": step_b,
                 "effective_GBps_cold": round(step_b / cold / 1e3, 1),
                 "effective_frac_of_peak_cold": round(step_b / cold / 1e3 / HBM_PEAK_GBS, 4),
                 "effective_GBps_warm": round(step_b / warm / 1e3, 1),
                 "speedup_vs_dense_cold": round(dense_cold / cold, 3),
                 "speedup_vs_dense_warm": round(dense_warm / warm, 3)}
        if is_primary:
            entry["warm_p10_p50_p90"] = warm_percentiles(args.steps)
            kt = kernel_times(args.steps)
            primary = (cold, warm, kt, kv_b, step_b, ub, dh, du, n_cold, entry)
        log(f"[bench] survival {s:.2f}: {entry}")
        sweep[f"{int(round(s * 100))}%"] = entry

    # ---- the no-screening arm: every block selected, dense gated attention (Eq. mult_attn
    # over all keys) through the same path, at the primary thresholds
    set_point(biases[PRIMARY_SURVIVAL])
    p_all = eta.decode_params(beta=wl.beta, z=wl.z, offset_a=wl.a, rescue_window=wl.rescue_window,
                              screen_all=True, num_splits=args.splits)
    st_all = eta.DecodeStep(q, k, v, sl, summ, W, bias_buf, block_size=bs, params=p_all)
    all_warm = time_warm(torch, st_all.run, max(20, args.steps // 4))
    all_cold = time_cold(torch, st_all.run, 20, flush)[0]
    screen_all = {"us_per_step_cold": all_cold, "us_per_step_warm": all_warm,
                  "union_blocks": int(st_all.union_counts.sum()),
                  "speedup_vs_dense_cold": round(dense_cold / all_cold, 3)}
    log(f"[bench] screen_all (dense gated): {screen_all}")
    del st_all

    # ---- the same steps screening on compact records (fp16 mu / sigma, the paper's
    # compact record; FP8 E4M3 mu / sigma, its FP8 metadata), with thresholds placed
    # from that index's own bounds (the same head survival); the headline keeps the
    # fp32 index
    def compact_index(stat_dtype, label):
        summ_c = eta.build_block_summaries(k, sl, bs, num_q_heads=Hq, stat_dtype=stat_dtype)
        bnd_c = eta.block_bounds(q, sl, summ_c, k, block_size=bs, z=wl.z).cpu().numpy()
        biases_c = {s: torch.as_tensor(place_bias(bnd_c, nblk, qW, s, wl.a), device=dev)
                    for s in SWEEP}
        prep_c = eta.DecodeStep(q, k, v, sl, summ_c, W, bias_buf, block_size=bs, params=params)
        res = {}
        for s in (SWEEP if not args.only_primary else (PRIMARY_SURVIVAL,)):
            set_point(biases_c[s])
            res[f"{int(round(s * 100))}%"] = {
                "warm": time_warm(torch, prep_c.run, max(20, args.steps // 4)),
                "cold": time_cold(torch, prep_c.run, 20, flush)[0]}
        set_point(biases_c[PRIMARY_SURVIVAL])
        eta.profile_begin()
        for _ in range(50):
            prep_c.run()
        torch.cuda.synchronize()
        kt_c = eta.profile_end()
        res["screen_avg_us_20%"] = round(kt_c["screen"][0] / max(kt_c["screen"][1], 1) * 1e3, 2)
        res["split_avg_us_20%"] = round(kt_c["split_decode"][0] / max(kt_c["split_decode"][1], 1) * 1e3, 2)
        log(f"[bench] {label} index: {res}")
        return res

    index_f16 = compact_index(torch.float16, "fp16")
    index_fp8 = compact_index(torch.float8_e4m3fn, "fp8")
    set_point(biases[PRIMARY_SURVIVAL])

    # ---- offline threshold calibration: 16 calibration sequences of 4096 steps at the
    # ragged workload's head shape (32 query / 8 kv heads, d = 128), 1024 bins
    calib = None
    if not args.no_calibration:
        from synth import calib_stream
        cN, cHq, cHkv, cT, cd, cnb = 16, 32, 8, 4096, 128, 1024
        cs = calib_stream(N=cN, Hq=cHq, Hkv=cHkv, T=cT, d=cd, seed=9, device=dev)
        cal = eta.Calibrator(cHq, cHkv, cd, beta=4.0, lo=-8.0, hi=24.0, num_bins=cnb, device=dev)
        cal.accumulate(cs.q, cs.k, cs.tau)        # warm-up
        torch.cuda.synchronize()
        cal.hist.zero_(); cal.density.zero_()
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record()
        cal.accumulate(cs.q, cs.k, cs.tau)
        e1.record()
        cal.solve()
        e2.record()
        torch.cuda.synchronize()
        acc_ms, solve_ms = e0.elapsed_time(e1), e1.elapsed_time(e2)
        pairs = cN * cHq * cT * (cT + 1) // 2
        flops = 2.0 * pairs * cd
        calib = {"workload": f"{cN} sequences x {cT} steps, {cHq}/{cHkv} heads, d={cd}, bf16, "
                             f"{cnb} bins",
                 "accumulate_ms": round(acc_ms, 3), "solve_us": round(solve_ms * 1e3, 1),
                 "causal_pairs_per_s": round(pairs / acc_ms * 1e3, 1),
                 "score_tflops": round(flops / acc_ms / 1e9, 1),
                 "score_frac_of_bf16_mfma_peak": round(flops / acc_ms / 1e9 / 2500.0, 4)}
        log(f"[bench] calibration: {calib}")
        del cs, cal

    # ---- gated prefill / training forward
    prefill = None if args.no_prefill else measure_prefill(torch, eta, dev)

    # ---- the other decode workloads at their library-default launch, each with its
    # dense baseline: 4K MHA fp32 (constant thresholds), 32K GQA (predictor ~10%),
    # 8 x 128K GQA (clustered + random planted blocks, predictor ~10%), 32 ragged
    # 16K-64K sequences at 32/8 heads (calibrated constants, and the predictor)
    others = None
    if not args.no_other_configs and not args.only_primary:
        from synth import config1, config2, config3, config5
        others = {}
        for name, mk, compact in (
                ("b1_4k_mha4_d64_blk64_fp32_constant", lambda: config1(device=dev), False),
                ("b1_32k_gqa16x4_d128_blk64_predictor", lambda: config2(device=dev), False),
                ("b8_128k_gqa16x4_d128_blk64_predictor", lambda: config3(device=dev), True),
                ("b32_ragged_16k_64k_gqa32x8_d128_blk64_constants", lambda: config5(device=dev), False),
                ("b32_ragged_16k_64k_gqa32x8_d128_blk64_predictor",
                 lambda: config5(device=dev, predictor=True), True)):
            owl = mk()
            others[name] = measure_config(torch, np, eta, dev, owl, 50, flush, compact)
            del owl
            torch.cuda.empty_cache()

    cold, warm, kt, kv_b, step_b, ub, dh, du, n_cold, pentry = primary
    split_ms, split_n = kt["split_decode"]
    split_avg_ms = split_ms / max(split_n, 1)
    achieved = kv_b / split_avg_ms / 1e6
    kernels = {name: {"avg_us": round(t / max(n, 1) * 1e3, 2), "launches": n}
               for name, (t, n) in kt.items() if n}

    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        try:
            tr = json.load(open(TRAFFIC_FILE))
            if tr.get("kernel_src_sha") == kernel_src_sha():
                traffic = tr.get("hbm_bytes_per_launch")
        except (ValueError, OSError):
            traffic = None

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, biases[PRIMARY_SURVIVAL], args.cpu_seconds)

    if args.copy_probe_mib > 0:
        src = torch.empty(args.copy_probe_mib << 20, dtype=torch.uint8, device=dev).fill_(3)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] copy probe: {args.copy_probe_mib} MiB copied")

    result = {
        "metric": "decode attention us/step + effective HBM GB/s (frac of peak) at 128K/512K ctx",
        "value": cold,
        "unit": "us/step",
        "n_gpus": 1,
        "steps": n_cold,
        "warmup": args.warmup,
        "ms_per_step": round(cold / 1e3, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "eta_decode_512k_b1_gqa16x4_d128_blk128_bf16_survival20",
                   "batch": B, "context": wl.seq_lens[0], "q_heads": Hq, "kv_heads": Hkv,
                   "head_dim": d, "block": bs, "survival_target": PRIMARY_SURVIVAL,
                   "beta": wl.beta, "z": wl.z, "rescue_window": wl.rescue_window,
                   "parallelism": "single_gpu"},
        "timing": "value = mean GPU time of one decode step after a 512 MiB read sweep "
                  "(last-level cache flushed; events around each step, the sweep outside them); "
                  "us_per_step_warm = back-to-back steps, wall clock",
        "cold_p10_p50_p90": pentry["cold_p10_p50_p90"],
        "us_per_step_warm": warm,
        "warm_p10_p50_p90": pentry["warm_p10_p50_p90"],
        "effective_GBps": round(step_b / cold / 1e3, 1),
        "effective_frac_of_peak": round(step_b / cold / 1e3 / HBM_PEAK_GBS, 4),
        "effective_GBps_warm": round(step_b / warm / 1e3, 1),
        "step_bytes": step_b,
        "d_head": round(dh, 4), "d_union": round(du, 4),
        "dense_us_per_step_cold": dense_cold, "dense_us_per_step_warm": dense_warm,
        "speedup_vs_dense": round(dense_cold / cold, 3),
        "speedup_vs_dense_warm": round(dense_warm / warm, 3),
        "screen_all_dense_gated": screen_all,
        "summary_build_us": round(sum_ms * 1e3, 1),
        "summary_build_GBps": round(sum_bytes / sum_ms / 1e6, 1),
        "summary_envelope_build_us": round(env_ms * 1e3, 1),
        "summary_envelope_sub_block": env_sub,
        "summary_update_us_per_step": round(upd_ms * 1e3, 2),
        "index_f16_us_per_step": index_f16,
        "index_fp8_us_per_step": index_fp8,
        "calibration": calib,
        "gated_prefill": prefill,
        "other_configs": others,
        "roofline": {"bound": "hbm", "kernel": "split_decode", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "algorithmic_bytes_per_launch": kv_b,
                     "avg_launch_us": round(split_avg_ms * 1e3, 2), "union_blocks": ub},
        "kernels": kernels,
        "cpu_baseline": cpu,
        "sweep": sweep,
        "paper_context": "up to 2.15x end-to-end decode speedup over FlashAttention-2 "
                         "(H100 SXM 80GB, fp16, 22-layer 1.45B model, B=64, 256K, 16% union)",
        "kernel_src_sha": kernel_src_sha(),
    }
    print(json.dumps(result), flush=True)


def cpu_baseline(wl, bias, budget_s):
    """The fp64 oracle (unchanged, OpenMP over heads) on this host, on the same step."""
    import numpy as np

    import oracle
    from synth import as_numpy

    log("[bench] cpu baseline: copying the workload to the host")
    q, k, v = as_numpy(wl.q), as_numpy(wl.k), as_numpy(wl.v)
    W = as_numpy(wl.W)
    b = bias.detach().cpu().numpy()
    t0 = time.perf_counter()
    summ = oracle.block_index(k, wl.seq_lens, wl.block)
    t_index = time.perf_counter() - t0
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
    rows = list(range(wl.B * wl.Hq))
    n, elapsed = 0, 0.0
    while True:
        t0 = time.perf_counter()
        tau = oracle.predict(q, W, b)
        oracle.decode(q, k, v, wl.seq_lens, tau, block_size=wl.block, beta=wl.beta, z=wl.z,
                      a=wl.a, rescue_window=wl.rescue_window, summaries=summ, rows=rows)
        elapsed += time.perf_counter() - t0
        n += 1
        if elapsed >= budget_s:
            break
    per_step_us = elapsed / n * 1e6
    log(f"[bench] cpu baseline {per_step_us:.0f} us/step over {n} steps "
        f"(block index {t_index:.1f} s, untimed)")
    # the same step on one thread (a few steps: ~0.4 s each), then the thread count back
    one_thread_us = None
    try:
        import ctypes
        gomp = ctypes.CDLL("libgomp.so.1")
        gomp.omp_set_num_threads(1)
        m, t1 = 0, 0.0
        while m < 2 or t1 < 1.0:
            t0 = time.perf_counter()
            tau = oracle.predict(q, W, b)
            oracle.decode(q, k, v, wl.seq_lens, tau, block_size=wl.block, beta=wl.beta, z=wl.z,
                          a=wl.a, rescue_window=wl.rescue_window, summaries=summ, rows=rows)
            t1 += time.perf_counter() - t0
            m += 1
        gomp.omp_set_num_threads(threads)
        one_thread_us = round(t1 / m * 1e6, 1)
        log(f"[bench] cpu baseline on one thread: {one_thread_us:.0f} us/step over {m} steps")
    except OSError:
        pass
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), None)
    except OSError:
        pass
    return {"value": round(per_step_us, 1), "unit": "us/step", "cores": min(threads, len(rows)),
            "kind": "oracle", "summary_build_s": round(t_index, 3),
            "sample": f"the full 512K step (all {len(rows)} query heads), repeated {n}x; "
                      f"block summaries precomputed by the oracle, untimed",
            "one_thread_us_per_step": one_thread_us, "cpu_model": cpu_model,
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


if __name__ == "__main__":
    main()
