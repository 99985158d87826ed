"""eta_decode_predicted_noalloc: the decode step with the library's own device
scratch instead of a caller's workspace (for callers that cannot allocate).

On the GPU its results must equal eta_decode_predicted's bit for bit, on
consecutive calls that leave each other's contents in the shared scratch (the
second call smaller than the first, then the first again).  On the host, a call
whose workspace would exceed the scratch is rejected before anything runs.
"""
import ctypes

import pytest
import torch

from gpu_support import calibrate_bias, require_gpu, say
from paper_2609_20888_amd import eta
from synth import make_workload

CASES = [
    dict(B=2, Hq=8, Hkv=2, d=128, block=64, seq_lens=[20000, 9001], planted={"frac": 0.05},
         predictor=True, target_survival=0.15, seed=81),
    dict(B=1, Hq=16, Hkv=4, d=128, block=128, seq_lens=[12345], planted={"frac": 0.03},
         predictor=True, target_survival=0.2, seed=82),
]


def _run_pair(kw):
    wl = make_workload(**kw)
    calibrate_bias(wl)
    dev = torch.device("cuda")
    q, k, v = wl.q.to(dev), wl.k.to(dev), wl.v.to(dev)
    sl = torch.tensor(wl.seq_lens, dtype=torch.int32, device=dev)
    summ = eta.build_block_summaries(k, sl, wl.block, num_q_heads=wl.Hq)
    W, bias = wl.W_heads.to(dev), wl.bias.to(dev)
    p = eta.decode_params(beta=wl.beta, z=wl.z, offset_a=wl.a, rescue_window=wl.rescue_window)
    tau_ref = torch.full((wl.B, wl.Hq), float("nan"), device=dev)
    ref = eta.decode_predicted(q, k, v, sl, summ, W, bias, block_size=wl.block, params=p,
                               tau_out=tau_ref)
    tau = torch.full_like(tau_ref, float("nan"))
    # outputs pre-filled with other values, so nothing stale can pass as a result
    got = eta.DecodeOut(out=torch.full_like(ref.out, 7.0),
                        mask=torch.full_like(ref.mask, 9),
                        counts=torch.full_like(ref.counts, -5),
                        union_counts=torch.full_like(ref.union_counts, -5))
    eta.decode_predicted_noalloc(q, k, v, sl, summ, W, bias, block_size=wl.block, params=p,
                                 out=got.out, mask=got.mask, counts=got.counts,
                                 union_counts=got.union_counts, tau_out=tau)
    torch.cuda.synchronize()
    for name in ("out", "mask", "counts", "union_counts"):
        assert torch.equal(getattr(got, name), getattr(ref, name)), name
    assert torch.equal(tau, tau_ref)
    return int(ref.union_counts.sum())


@pytest.mark.gpu
def test_noalloc_equals_decode_predicted_on_consecutive_calls():
    require_gpu()
    for i in (0, 1, 0):
        u = _run_pair(CASES[i])
        say(f"[gpu] noalloc case {i}: bit-identical to eta_decode_predicted ({u} union blocks)")


def test_noalloc_rejects_calls_beyond_the_scratch():
    lib = eta.load_library()
    FAKE = 0x10000
    # 8 sequences x 64 query heads x 1024 splits x 128 dims of fp32 partials: 268 MB
    desc = eta.KvDesc(batch=8, num_q_heads=64, num_kv_heads=8, head_dim=128, block_size=64,
                      kv_dtype=eta.ETA_DT_BF16, capacity_tokens=4096, stride_b=8 * 4096 * 128,
                      stride_h=4096 * 128, stride_t=128)
    summ = eta.SummaryDesc(mu=FAKE, sigma=FAKE, max_norm=FAKE, n_blk_cap=64)
    p = eta.decode_params(num_splits=1024)
    need = eta.decode_workspace_size(desc, summ.n_blk_cap, p)
    assert need > eta.NOALLOC_SCRATCH_BYTES
    st = lib.eta_decode_predicted_noalloc(ctypes.byref(desc), eta.ETA_DT_BF16, FAKE, FAKE, FAKE,
                                          FAKE, ctypes.byref(summ), FAKE, FAKE, ctypes.byref(p),
                                          FAKE, FAKE, None, None, None, None)
    assert st == eta.ETA_ERR_WORKSPACE
    msg = lib.eta_last_error_string().decode()
    assert str(need) in msg and str(eta.NOALLOC_SCRATCH_BYTES) in msg
    # argument errors are reported before the size
    assert lib.eta_decode_predicted_noalloc(ctypes.byref(desc), eta.ETA_DT_BF16, FAKE, FAKE, FAKE,
                                            FAKE, ctypes.byref(summ), FAKE, None, ctypes.byref(p),
                                            FAKE, FAKE, None, None, None, None) \
        == eta.ETA_ERR_INVALID_ARG
