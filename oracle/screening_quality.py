"""Screening-quality table of the synthetic decode workloads (test infrastructure).

    python -m oracle.screening_quality [--out oracle/screening_quality.json]

For each workload the benchmark and the parity tests use (the 4K MHA fp32, 32K
GQA, 8 x 128K GQA, 512K GQA at the four survival points, and the 32 ragged
sequences with constant and with predicted thresholds), draws the seeded
inputs on the CPU, places the predictor bias from the oracle's own bounds
(synth.place_bias) where the workload uses the predictor, and runs the oracle's
decode with its screening-quality diagnostics (Tab. "index_quality"): block
false-negative and false-positive rates, recall of above-threshold keys, the
missed gated softmax mass, and the head / GQA-union densities.  Only the
oracle and the seeded input generators are used; the GPU library is not.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from synth import as_numpy, config1, config2, config3, config4, config5, place_bias  # noqa: E402


def evaluate(wl, survival=None):
    q, k, v = as_numpy(wl.q), as_numpy(wl.k), as_numpy(wl.v)
    summ = oracle.block_index(k, wl.seq_lens, wl.block)
    nb = [t // wl.block for t in wl.seq_lens]
    if wl.W is not None:
        W = as_numpy(wl.W)
        r0 = oracle.decode(q, k, v, wl.seq_lens, None, block_size=wl.block, z=wl.z,
                           bounds_only=True, summaries=summ)
        qW = oracle.predict(q, W, None)
        target = survival if survival is not None else wl.target_survival
        bias = place_bias(r0.bounds, nb, qW, target, wl.a)
        tau = oracle.predict(q, W, bias)
    else:
        tau = oracle.predict(q, None, as_numpy(wl.bias))
    r = oracle.decode(q, k, v, wl.seq_lens, tau, block_size=wl.block, beta=wl.beta, z=wl.z,
                      a=wl.a, rescue_window=wl.rescue_window, lwb=wl.lwb, summaries=summ,
                      quality=True)
    rates = oracle.quality_rates(r)
    G = wl.Hq // wl.Hkv
    head = sum(int(r.sel[b, :, :nb[b]].sum()) for b in range(wl.B))
    union = sum(int(r.sel[b, g * G:(g + 1) * G, :nb[b]].any(axis=0).sum())
                for b in range(wl.B) for g in range(wl.Hkv))
    rates["d_head"] = head / float(wl.Hq * sum(nb))
    rates["d_union"] = union / float(wl.Hkv * sum(nb))
    rates["rescued_rows"] = int(np.count_nonzero(r.rescued >= 0))
    return rates


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=os.path.join(HERE, "screening_quality.json"))
    args = ap.parse_args()
    runs = [("4K MHA fp32, tau 2.0, z 1", lambda: config1(), None),
            ("32K GQA 16/4, predictor ~10%, z 1", lambda: config2(), None),
            ("8 x 128K GQA 16/4, predictor ~10%, z 1", lambda: config3(), None)]
    runs += [(f"512K GQA 16/4, predictor {int(s * 100)}%, z 1", lambda: config4(), s)
             for s in (0.01, 0.05, 0.20, 1.00)]
    runs += [("32 ragged 16K-64K, 32/8, constants U[1.5, 3], z 2", lambda: config5(), None),
             ("32 ragged 16K-64K, 32/8, predictor ~10%, z 2", lambda: config5(predictor=True), None)]
    table = []
    cache = {}
    for name, make, surv in runs:
        t0 = time.perf_counter()
        wl = cache.get("c4") if surv is not None else None
        if wl is None:
            wl = make()
            if surv is not None:
                cache["c4"] = wl
        rates = evaluate(wl, surv)
        rates["workload"] = name
        table.append(rates)
        print(f"{name}: {json.dumps({k: (round(v, 5) if isinstance(v, float) else v) for k, v in rates.items() if k != 'workload'})} "
              f"({time.perf_counter() - t0:.0f} s)", flush=True)
        if surv is None:
            del wl
    with open(args.out, "w") as f:
        json.dump({"generator": "synth (CPU torch generator, seeded as in the tests)",
                   "definitions": {
                       "false_negative_rate": "full blocks whose brute-force max score >= tau_eff that are not selected / such blocks",
                       "false_positive_rate": "selected blocks whose max score < tau_eff / selected blocks",
                       "token_recall": "attended full-block keys with score >= tau_eff / full-block keys with score >= tau_eff",
                       "missed_mass": "gated softmax mass of the rejected blocks over all keys (mean and largest row)"},
                   "rows": table}, f, indent=1)
    print(f"wrote {args.out}")


if __name__ == "__main__":
    main()
