"""GPU parity of the gated prefill / training forward (App. "Hardware-Aligned
Forward Kernel") against the oracle; needs an MI355X.

Outputs per (sequence, head) row: max_c |o_gpu - o_ref| / max |o_ref| over a
head's rows (over the row, for sampled rows) <= 2e-2 (bf16 operands, softmax weights rounded to bf16 for p.V);
gate row sums R to 1e-4 relative (fp32 sums of gates whose scores differ from
fp64 by fp32 accumulation); log-sum-exp L to 1e-4 absolute.  Rows past a
sequence's length are zero / 0 / -inf.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_support import require_gpu, say
from paper_2609_20888_amd import eta
from synth import as_numpy

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu(request):
    require_gpu()
    say(f"\n[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


def _inputs(B, Hq, Hkv, T, d, seed, tau_mode="normal", q_scale=1.0):
    gen = torch.Generator().manual_seed(seed)
    q = (q_scale * torch.randn(B, Hq, T, d, generator=gen)).to(torch.bfloat16)
    k = torch.randn(B, Hkv, T, d, generator=gen).to(torch.bfloat16)
    v = torch.randn(B, Hkv, T, d, generator=gen).to(torch.bfloat16)
    if tau_mode == "normal":
        tau = 0.5 + 0.5 * torch.randn(B, Hq, T, generator=gen)
    elif tau_mode == "ungated":
        tau = torch.full((B, Hq, T), float("-inf"))
    else:
        tau = torch.full((B, Hq, T), float("inf"))
    return q, k, v, tau.float()


CASES = {
    # name: (B, Hq, Hkv, T, d, seq_lens, beta, additive, C, tau_mode)
    "gqa2_d128_ragged": (2, 4, 2, 200, 128, [200, 131], 4.0, False, 0.0, "normal"),
    "gqa8_d64": (1, 8, 1, 256, 64, [256], 4.0, False, 0.0, "normal"),
    "mha_d128_additive": (1, 2, 2, 160, 128, [150], 2.0, True, 3.0, "normal"),
    "ungated_is_causal_softmax": (1, 4, 4, 130, 64, [130], 4.0, False, 0.0, "ungated"),
    "closed_gates_diagonal_only": (1, 4, 2, 96, 128, [96], 4.0, False, 0.0, "closed"),
    "short_and_empty": (3, 4, 2, 70, 128, [1, 0, 65], 4.0, False, 0.0, "normal"),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_prefill_matches_oracle(name):
    B, Hq, Hkv, T, d, lens, beta, add, C, tm = CASES[name]
    q, k, v, tau = _inputs(B, Hq, Hkv, T, d, seed=hash(name) % 1000, tau_mode=tm)
    dev = torch.device("cuda")
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    out, R, L = eta.gated_prefill(q.to(dev), k.to(dev), v.to(dev), tau.to(dev), sl, beta=beta,
                                  additive=add, C=C)
    torch.cuda.synchronize()
    r = oracle.prefill(as_numpy(q), as_numpy(k), as_numpy(v), tau.numpy().astype(np.float64), lens,
                       beta=beta, additive=add, C=C)
    o = out.float().cpu().numpy()
    Rg, Lg = R.cpu().numpy(), L.cpu().numpy()
    worst = 0.0
    for b in range(B):
        n = lens[b]
        assert np.all(o[b, :, n:] == 0) and np.all(Rg[b, :, n:] == 0) and np.all(np.isneginf(Lg[b, :, n:]))
        if n == 0:
            continue
        for h in range(Hq):
            ref = r.o[b, h, :n]
            err = float(np.max(np.abs(o[b, h, :n] - ref)) / np.max(np.abs(ref)))
            worst = max(worst, err)
            assert err <= 2e-2, (b, h, err)
        np.testing.assert_allclose(Rg[b, :, :n], r.r[b, :, :n], rtol=1e-4, atol=1e-5)
        np.testing.assert_allclose(Lg[b, :, :n], r.lse[b, :, :n], rtol=0, atol=1e-4)
    say(f"[gpu] prefill {name}: worst output rel err {worst:.2e}")


def _check_rows(o, R, L, r, rows, lens):
    worst = 0.0
    for n, (b, h, i) in enumerate(rows):
        if i >= lens[b]:
            assert np.all(o[n] == 0) and R[n] == 0 and np.isneginf(L[n])
            continue
        err = float(np.max(np.abs(o[n] - r.o[n])) / np.max(np.abs(r.o[n])))
        worst = max(worst, err)
        assert err <= 2e-2, (b, h, i, err)
        np.testing.assert_allclose(R[n], r.r[n], rtol=1e-4, atol=1e-5, err_msg=str((b, h, i)))
        np.testing.assert_allclose(L[n], r.lse[n], rtol=0, atol=1e-4, err_msg=str((b, h, i)))
    return worst


def test_prefill_long_rows_with_rescaling():
    """1100 tokens (9 query tiles, 18 key blocks, a ragged end) with queries scaled
    up so that the row maxima keep growing and the running reference moves often;
    both gate forms."""
    B, Hq, Hkv, T, d, lens = 1, 4, 1, 1100, 128, [1037]
    q, k, v, tau = _inputs(B, Hq, Hkv, T, d, seed=321, q_scale=3.0)
    dev = torch.device("cuda")
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    rng = np.random.default_rng(5)
    rows = np.array([[0, h, i] for h in range(Hq)
                     for i in sorted({0, 63, 64, 127, 128, 1023, 1036, 1037, 1099}
                                     | set(rng.integers(0, T, 24).tolist()))])
    for add, C in ((False, 0.0), (True, 4.0)):
        out, R, L = eta.gated_prefill(q.to(dev), k.to(dev), v.to(dev), tau.to(dev), sl, beta=4.0,
                                      additive=add, C=C)
        torch.cuda.synchronize()
        r = oracle.prefill_rows(as_numpy(q), as_numpy(k), as_numpy(v),
                                tau.numpy().astype(np.float64), lens, rows, beta=4.0,
                                additive=add, C=C)
        idx = tuple(rows.T)
        worst = _check_rows(out.float().cpu().numpy()[idx], R.cpu().numpy()[idx],
                            L.cpu().numpy()[idx], r, rows, lens)
        say(f"[gpu] prefill long additive={add}: worst output rel err {worst:.2e}")


def test_prefill_full_size_sampled_rows():
    """The benchmarked prefill workload (16384 tokens, 32 query / 8 KV heads, d=128,
    bf16, causal) in the same launch, checked on sampled rows: tile edges, the first
    and last rows, and random rows of every head."""
    B, Hq, Hkv, T, d, lens = 1, 32, 8, 16384, 128, [16384]
    say("[gpu] prefill full size: building inputs")
    q, k, v, tau = _inputs(B, Hq, Hkv, T, d, seed=2024)
    dev = torch.device("cuda")
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    out, R, L = eta.gated_prefill(q.to(dev), k.to(dev), v.to(dev), tau.to(dev), sl, beta=4.0)
    torch.cuda.synchronize()
    rng = np.random.default_rng(6)
    fixed = [0, 1, 63, 64, 127, 128, 4095, 8192, 16255, 16256, 16383]
    rows = np.array([[0, h, i] for h in range(Hq)
                     for i in sorted(set(fixed[h % 4::4]) | set(rng.integers(0, T, 3).tolist()))])
    say(f"[gpu] prefill full size: oracle on {len(rows)} rows")
    r = oracle.prefill_rows(as_numpy(q), as_numpy(k), as_numpy(v), tau.numpy().astype(np.float64),
                            lens, rows, beta=4.0)
    idx = tuple(rows.T)
    worst = _check_rows(out.float().cpu().numpy()[idx], R.cpu().numpy()[idx], L.cpu().numpy()[idx],
                        r, rows, lens)
    say(f"[gpu] prefill full size: worst output rel err {worst:.2e} over {len(rows)} rows")
