"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments on the host before any launch."""
import ctypes
import os
import re

import pytest
import torch

from paper_2609_20888_amd import eta

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "eta.h")


@pytest.fixture(scope="module")
def lib():
    return eta.load_library()


def test_header_declarations_are_all_exported(lib):
    text = open(HEADER).read()
    declared = set(re.findall(r"^\s*(?:eta_status_t|const char\*|int32_t)\s+(eta_\w+)\s*\(", text, re.M))
    assert declared == set(eta.EXPORTS), declared ^ set(eta.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name
    assert lib.eta_abi_version() == 5


def good_desc(**kw):
    d = dict(batch=1, num_q_heads=16, num_kv_heads=4, head_dim=128, block_size=64,
             kv_dtype=eta.ETA_DT_BF16, capacity_tokens=4096, stride_b=4 * 4096 * 128,
             stride_h=4096 * 128, stride_t=128)
    d.update(kw)
    return eta.KvDesc(**d)


def ws_size(lib, desc, params, n_blk_cap=None):
    if n_blk_cap is None:
        n_blk_cap = max(max(desc.capacity_tokens, 0) // max(desc.block_size, 1), 1)
    n = ctypes.c_size_t()
    st = lib.eta_decode_workspace_size(ctypes.byref(desc), n_blk_cap, ctypes.byref(params),
                                       ctypes.byref(n))
    return st, n.value


def test_workspace_size_valid_and_monotone(lib):
    p = eta.decode_params()
    st, n1 = ws_size(lib, good_desc(), p)
    assert st == eta.ETA_OK and n1 > 0 and n1 % 256 == 0
    st, n2 = ws_size(lib, good_desc(capacity_tokens=8192), p)
    assert st == eta.ETA_OK and n2 > n1
    st, n3 = ws_size(lib, good_desc(), eta.decode_params(num_splits=512))
    assert st == eta.ETA_OK and n3 > n1
    # the workspace follows the summary's block capacity, which may exceed the cache's
    st, n4 = ws_size(lib, good_desc(), p, n_blk_cap=4096 // 64 + 64)
    assert st == eta.ETA_OK and n4 > n1
    st, n5 = ws_size(lib, good_desc(capacity_tokens=52), p, n_blk_cap=1)
    assert st == eta.ETA_OK and n5 > 0
    # a summary holds at least one block, also below one block of capacity
    assert ws_size(lib, good_desc(capacity_tokens=52), p, n_blk_cap=0)[0] == eta.ETA_ERR_INVALID_ARG
    assert ws_size(lib, good_desc(), p, n_blk_cap=4096 // 64 - 1)[0] == eta.ETA_ERR_INVALID_ARG
    assert ws_size(lib, good_desc(), p, n_blk_cap=131073)[0] == eta.ETA_ERR_UNSUPPORTED


@pytest.mark.parametrize("kw,code", [
    (dict(batch=0), eta.ETA_ERR_INVALID_ARG),
    (dict(num_kv_heads=3), eta.ETA_ERR_INVALID_ARG),             # 16 % 3 != 0
    (dict(num_q_heads=32, num_kv_heads=2), eta.ETA_ERR_UNSUPPORTED),  # G = 16
    (dict(head_dim=96, stride_t=96), eta.ETA_ERR_UNSUPPORTED),
    (dict(block_size=32), eta.ETA_ERR_UNSUPPORTED),
    (dict(capacity_tokens=0), eta.ETA_ERR_INVALID_ARG),
    (dict(kv_dtype=7), eta.ETA_ERR_INVALID_ARG),
    (dict(stride_t=100), eta.ETA_ERR_INVALID_ARG),                # < head_dim
    (dict(stride_t=132), eta.ETA_ERR_INVALID_ARG),                # rows not 16-byte aligned
    (dict(stride_h=-1), eta.ETA_ERR_INVALID_ARG),
])
def test_geometry_rejected(lib, kw, code):
    st, _ = ws_size(lib, good_desc(**kw), eta.decode_params())
    assert st == code
    assert lib.eta_last_error_string().decode() != ""


@pytest.mark.parametrize("kw,code", [
    (dict(beta=float("nan")), eta.ETA_ERR_INVALID_ARG),
    (dict(beta=-1.0), eta.ETA_ERR_INVALID_ARG),
    (dict(z=float("inf")), eta.ETA_ERR_INVALID_ARG),
    (dict(offset_a=float("nan")), eta.ETA_ERR_INVALID_ARG),
    (dict(rescue_window=-1), eta.ETA_ERR_INVALID_ARG),
    (dict(rescue_window=257), eta.ETA_ERR_UNSUPPORTED),
    (dict(lwb=-2), eta.ETA_ERR_INVALID_ARG),
    (dict(num_splits=2000), eta.ETA_ERR_INVALID_ARG),
])
def test_params_rejected(lib, kw, code):
    st, _ = ws_size(lib, good_desc(), eta.decode_params(**kw))
    assert st == code


FAKE = 0x10000          # aligned, never dereferenced: validation fails first or nothing launches


def decode_call(lib, desc=None, q=FAKE, tau=FAKE, out=FAKE, mask=FAKE, ws=FAKE, ws_bytes=1 << 30,
                summ=None, params=None):
    desc = desc or good_desc()
    summ = summ or eta.SummaryDesc(mu=FAKE, sigma=FAKE, max_norm=FAKE, n_blk_cap=64)
    params = params or eta.decode_params()
    return lib.eta_decode(ctypes.byref(desc), eta.ETA_DT_BF16, q, FAKE, FAKE, FAKE,
                          ctypes.byref(summ), tau, ctypes.byref(params), out, mask, None, None,
                          ws, ws_bytes, None)


def test_decode_rejects_null_and_misaligned(lib):
    assert decode_call(lib, q=None) == eta.ETA_ERR_INVALID_ARG
    assert decode_call(lib, tau=None) == eta.ETA_ERR_INVALID_ARG
    assert decode_call(lib, mask=None) == eta.ETA_ERR_INVALID_ARG
    assert decode_call(lib, out=FAKE + 2) == eta.ETA_ERR_INVALID_ARG
    assert "aligned" in lib.eta_last_error_string().decode()


def test_decode_rejects_workspace_problems(lib):
    assert decode_call(lib, ws=None) == eta.ETA_ERR_WORKSPACE
    assert decode_call(lib, ws=FAKE + 16) == eta.ETA_ERR_WORKSPACE
    assert decode_call(lib, ws_bytes=100) == eta.ETA_ERR_WORKSPACE
    assert "too small" in lib.eta_last_error_string().decode()


def test_decode_rejects_small_summary_capacity(lib):
    s = eta.SummaryDesc(mu=FAKE, sigma=FAKE, max_norm=FAKE, n_blk_cap=63)   # 4096 / 64 = 64 needed
    assert decode_call(lib, summ=s) == eta.ETA_ERR_INVALID_ARG
    s = eta.SummaryDesc(mu=None, sigma=FAKE, max_norm=FAKE, n_blk_cap=64)
    assert decode_call(lib, summ=s) == eta.ETA_ERR_INVALID_ARG


def test_predict_rejects(lib):
    f = lib.eta_predict_threshold
    assert f(0, 16, 128, eta.ETA_DT_BF16, FAKE, None, FAKE, FAKE, None) == eta.ETA_ERR_INVALID_ARG
    assert f(1, 300, 128, eta.ETA_DT_BF16, FAKE, None, FAKE, FAKE, None) == eta.ETA_ERR_UNSUPPORTED
    assert f(1, 16, 128, 5, FAKE, None, FAKE, FAKE, None) == eta.ETA_ERR_INVALID_ARG
    assert f(1, 16, 128, eta.ETA_DT_BF16, FAKE, None, None, FAKE, None) == eta.ETA_ERR_INVALID_ARG


def test_dense_and_bounds_reject(lib):
    d = good_desc()
    n = ctypes.c_size_t()
    assert lib.eta_dense_workspace_size(ctypes.byref(d), -1, ctypes.byref(n)) == eta.ETA_ERR_INVALID_ARG
    assert lib.eta_dense_workspace_size(ctypes.byref(d), 0, ctypes.byref(n)) == eta.ETA_OK
    assert lib.eta_dense_decode(ctypes.byref(d), eta.ETA_DT_BF16, FAKE, FAKE, FAKE, FAKE, FAKE, 0,
                                None, 1 << 20, None) == eta.ETA_ERR_WORKSPACE
    s = eta.SummaryDesc(mu=FAKE, sigma=FAKE, max_norm=FAKE, n_blk_cap=64)
    assert lib.eta_block_bounds(ctypes.byref(d), eta.ETA_DT_BF16, FAKE, FAKE, ctypes.byref(s),
                                ctypes.c_float(-1.0), FAKE, None) == eta.ETA_ERR_INVALID_ARG


def test_profile_roundtrip_without_launches(lib):
    assert lib.eta_profile_begin() == eta.ETA_OK
    arr = (eta.KernelTime * len(eta.KERNEL_KINDS))()
    assert lib.eta_profile_end(arr) == eta.ETA_OK
    assert all(arr[i].launches == 0 for i in range(len(eta.KERNEL_KINDS)))


def test_summary_variants_reject(lib):
    d = good_desc()                                  # block_size 64
    s = eta.SummaryDesc(mu=FAKE, sigma=FAKE, max_norm=FAKE, n_blk_cap=64)
    env = lib.eta_build_block_summaries_envelope
    for bad in (-1, 3, 48, 128):                     # not a power of two in [1, 64]
        assert env(ctypes.byref(d), FAKE, FAKE, bad, ctypes.byref(s), None) == eta.ETA_ERR_INVALID_ARG
    assert "sub_block" in lib.eta_last_error_string().decode()
    upd = lib.eta_update_block_summaries
    assert upd(ctypes.byref(d), FAKE, None, FAKE, 1, 0, ctypes.byref(s), None) == eta.ETA_ERR_INVALID_ARG
    assert upd(ctypes.byref(d), FAKE, FAKE, FAKE, -1, 0, ctypes.byref(s), None) == eta.ETA_ERR_INVALID_ARG
    assert upd(ctypes.byref(d), FAKE, FAKE + 4, FAKE, 1, 0, ctypes.byref(s), None) == eta.ETA_ERR_INVALID_ARG
    assert upd(ctypes.byref(d), FAKE, FAKE, FAKE, 1, 5, ctypes.byref(s), None) == eta.ETA_ERR_INVALID_ARG
    small = eta.SummaryDesc(mu=FAKE, sigma=FAKE, max_norm=FAKE, n_blk_cap=63)
    assert upd(ctypes.byref(d), FAKE, FAKE, FAKE, 1, 0, ctypes.byref(small), None) == eta.ETA_ERR_INVALID_ARG
    # no block can have completed: nothing is launched
    assert upd(ctypes.byref(d), FAKE, FAKE, FAKE, 0, 4, ctypes.byref(s), None) == eta.ETA_OK


def test_summary_stat_dtypes_accepted(lib):
    """fp32, fp16 and FP8 (E4M3) records pass validation (an update with no block
    to write launches nothing and returns OK)."""
    d = good_desc()
    for ok in (eta.ETA_DT_F32, eta.ETA_DT_F16, eta.ETA_DT_FP8):
        s = eta.SummaryDesc(mu=FAKE, sigma=FAKE, max_norm=FAKE, n_blk_cap=64, stat_dtype=ok)
        assert lib.eta_update_block_summaries(ctypes.byref(d), FAKE, FAKE, FAKE, 0, 0,
                                              ctypes.byref(s), None) == eta.ETA_OK


def test_summary_stat_dtype_rejected(lib):
    d = good_desc()
    for bad in (eta.ETA_DT_BF16, 7):
        s = eta.SummaryDesc(mu=FAKE, sigma=FAKE, max_norm=FAKE, n_blk_cap=64, stat_dtype=bad)
        assert lib.eta_build_block_summaries(ctypes.byref(d), FAKE, FAKE, ctypes.byref(s), None) \
            == eta.ETA_ERR_INVALID_ARG
        assert "stat_dtype" in lib.eta_last_error_string().decode()
        assert decode_call(lib, summ=s) == eta.ETA_ERR_INVALID_ARG


def test_calibration_rejects(lib):
    def desc(**kw):
        d = dict(num_seqs=2, num_q_heads=8, num_kv_heads=2, head_dim=128, seq_len=256,
                 dtype=eta.ETA_DT_BF16, beta=4.0, lo=-4.0, hi=4.0, num_bins=512)
        d.update(kw)
        return eta.CalibDesc(**d)
    st = eta.CalibState(hist=FAKE, density=FAKE)
    acc = lambda cd, s=st, q=FAKE, k=FAKE, t=FAKE: lib.eta_calib_accumulate(
        ctypes.byref(cd), q, k, t, ctypes.byref(s), None)
    bad = [(dict(num_seqs=0), eta.ETA_ERR_INVALID_ARG), (dict(seq_len=0), eta.ETA_ERR_INVALID_ARG),
           (dict(num_kv_heads=3), eta.ETA_ERR_INVALID_ARG), (dict(num_kv_heads=1, num_q_heads=16), eta.ETA_ERR_UNSUPPORTED),
           (dict(head_dim=96), eta.ETA_ERR_UNSUPPORTED), (dict(dtype=eta.ETA_DT_F32), eta.ETA_ERR_UNSUPPORTED),
           (dict(beta=0.0), eta.ETA_ERR_INVALID_ARG), (dict(beta=float("nan")), eta.ETA_ERR_INVALID_ARG),
           (dict(lo=1.0, hi=1.0), eta.ETA_ERR_INVALID_ARG), (dict(hi=float("inf")), eta.ETA_ERR_INVALID_ARG),
           (dict(num_bins=0), eta.ETA_ERR_INVALID_ARG), (dict(num_bins=4097), eta.ETA_ERR_INVALID_ARG),
           (dict(num_seqs=64, seq_len=1 << 17), eta.ETA_ERR_INVALID_ARG)]
    for kw, code in bad:
        assert acc(desc(**kw)) == code, kw
    assert acc(desc(), q=None) == eta.ETA_ERR_INVALID_ARG
    assert acc(desc(), t=FAKE + 4) == eta.ETA_ERR_INVALID_ARG
    assert acc(desc(), s=eta.CalibState(hist=None, density=FAKE)) == eta.ETA_ERR_INVALID_ARG
    assert acc(desc(), s=eta.CalibState(hist=FAKE + 4, density=FAKE)) == eta.ETA_ERR_INVALID_ARG
    assert lib.eta_calib_solve(ctypes.byref(desc()), ctypes.byref(st), None, None, None) \
        == eta.ETA_ERR_INVALID_ARG


def test_prefill_rejects(lib):
    def desc(**kw):
        d = dict(batch=1, num_q_heads=8, num_kv_heads=2, head_dim=128, capacity_tokens=256,
                 dtype=eta.ETA_DT_BF16, beta=4.0, additive=0, C=0.0)
        d.update(kw)
        return eta.PrefillDesc(**d)
    call = lambda pd, **p: lib.eta_gated_prefill(
        ctypes.byref(pd), p.get("q", FAKE), FAKE, FAKE, p.get("tau", FAKE), FAKE, p.get("out", FAKE),
        FAKE, FAKE, None)
    for kw, code in [(dict(batch=0), eta.ETA_ERR_INVALID_ARG), (dict(capacity_tokens=0), eta.ETA_ERR_INVALID_ARG),
                     (dict(num_kv_heads=3), eta.ETA_ERR_INVALID_ARG), (dict(head_dim=80), eta.ETA_ERR_UNSUPPORTED),
                     (dict(num_kv_heads=1, num_q_heads=16), eta.ETA_ERR_UNSUPPORTED),
                     (dict(dtype=eta.ETA_DT_F32), eta.ETA_ERR_UNSUPPORTED), (dict(beta=-1.0), eta.ETA_ERR_INVALID_ARG),
                     (dict(additive=2), eta.ETA_ERR_INVALID_ARG), (dict(additive=1, C=float("inf")), eta.ETA_ERR_INVALID_ARG)]:
        assert call(desc(**kw)) == code, kw
    assert call(desc(), q=None) == eta.ETA_ERR_INVALID_ARG
    assert call(desc(), out=FAKE + 8) == eta.ETA_ERR_INVALID_ARG
    assert call(desc(), tau=FAKE + 2) == eta.ETA_ERR_INVALID_ARG


def test_binding_checks_predictor_layout():
    # the C ABI sees only pointers: the binding refuses a W that is not fp32
    # [Hq][Hq d] contiguous (the head-major layout) before any call
    q = torch.zeros(2, 4, 8, dtype=torch.bfloat16)
    bias = torch.zeros(4)
    for W in (torch.zeros(32, 4),                   # the [Hq d][Hq] layout
              torch.zeros(4, 32, dtype=torch.float64),
              torch.zeros(32, 4).t(),               # head-major shape, not contiguous
              torch.zeros(4, 31)):
        with pytest.raises(ValueError):
            eta.predict_threshold(q, W, bias)
    with pytest.raises(ValueError):
        eta.predict_threshold(q, torch.zeros(4, 32), torch.zeros(5))
