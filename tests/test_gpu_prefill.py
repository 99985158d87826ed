"""GPU parity of the gated prefill / training forward (App. "Hardware-Aligned
Forward Kernel") against the oracle; needs an MI355X.

Outputs per (sequence, head) row: max_c |o_gpu - o_ref| / max |o_ref| over a
head's rows <= 2e-2 (bf16 operands, softmax weights rounded to bf16 for p.V);
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


def _inputs(B, Hq, Hkv, T, d, seed, tau_mode="normal"):
    gen = torch.Generator().manual_seed(seed)
    q = torch.randn(B, Hq, T, d, generator=gen).to(torch.bfloat16)
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
