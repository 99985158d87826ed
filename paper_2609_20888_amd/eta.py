"""Python binding of libeta (include/eta.h): argument marshalling only.

Every function here hands torch tensors' device pointers and the current HIP
stream to the C ABI of the same name; all computation runs in the library's
HIP kernels.  There is no fallback: if ``libeta.so`` is missing or a call
fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libeta.so")

ETA_OK, ETA_ERR_INVALID_ARG, ETA_ERR_UNSUPPORTED, ETA_ERR_WORKSPACE, ETA_ERR_HIP = range(5)
ETA_DT_F32, ETA_DT_BF16, ETA_DT_F16, ETA_DT_FP8 = 0, 1, 2, 3
KERNEL_KINDS = ("summaries", "predict", "screen", "split_decode", "combine", "dense_split",
                "dense_combine", "bounds", "calib_accumulate", "calib_solve", "prefill")

_vp = ctypes.c_void_p


class KvDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("kv_dtype", ctypes.c_int32),
                ("capacity_tokens", ctypes.c_int64),
                ("stride_b", ctypes.c_int64), ("stride_h", ctypes.c_int64),
                ("stride_t", ctypes.c_int64)]


class SummaryDesc(ctypes.Structure):
    _fields_ = [("mu", _vp), ("sigma", _vp), ("max_norm", _vp), ("n_blk_cap", ctypes.c_int64),
                ("stat_dtype", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class CalibDesc(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("seq_len", ctypes.c_int32), ("dtype", ctypes.c_int32), ("beta", ctypes.c_float),
                ("lo", ctypes.c_float), ("hi", ctypes.c_float), ("num_bins", ctypes.c_int32)]


class CalibState(ctypes.Structure):
    _fields_ = [("hist", _vp), ("density", _vp)]


class PrefillDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("capacity_tokens", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("beta", ctypes.c_float), ("additive", ctypes.c_int32), ("C", ctypes.c_float)]


class DecodeParams(ctypes.Structure):
    _fields_ = [("beta", ctypes.c_float), ("z", ctypes.c_float), ("offset_a", ctypes.c_float),
                ("rescue_window_blocks", ctypes.c_int32), ("pin_recent_blocks", ctypes.c_int32),
                ("self_ungated", ctypes.c_int32), ("screen_all", ctypes.c_int32),
                ("num_splits", ctypes.c_int32)]


class KernelTime(ctypes.Structure):
    _fields_ = [("ms_total", ctypes.c_double), ("launches", ctypes.c_int64)]


# Symbols include/eta.h declares (the CPU test checks the library exports each).
EXPORTS = ("eta_build_block_summaries", "eta_build_block_summaries_envelope",
           "eta_update_block_summaries", "eta_predict_threshold", "eta_decode_workspace_size",
           "eta_decode", "eta_decode_predicted", "eta_decode_predicted_noalloc", "eta_block_bounds", "eta_dense_workspace_size", "eta_dense_decode",
           "eta_calib_accumulate", "eta_calib_solve", "eta_gated_prefill",
           "eta_last_error_string", "eta_abi_version", "eta_profile_begin", "eta_profile_end")


class EtaError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"libeta status {status}: {msg}")
        self.status = status


_lib = None


def load_library(path: Optional[str] = None):
    """Load libeta.so (built by ``paper_2609_20888_amd.build``); raise if it is missing."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is not built: run `python -m paper_2609_20888_amd.build` "
                           "(there is no non-HIP fallback)")
    lib = ctypes.CDLL(p)
    P = ctypes.POINTER
    i32, i64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    sz = ctypes.c_size_t
    sigs = {
        "eta_build_block_summaries": [P(KvDesc), _vp, _vp, P(SummaryDesc), _vp],
        "eta_calib_accumulate": [P(CalibDesc), _vp, _vp, _vp, P(CalibState), _vp],
        "eta_calib_solve": [P(CalibDesc), P(CalibState), _vp, _vp, _vp],
        "eta_gated_prefill": [P(PrefillDesc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp],
        "eta_build_block_summaries_envelope": [P(KvDesc), _vp, _vp, i32, P(SummaryDesc), _vp],
        "eta_update_block_summaries": [P(KvDesc), _vp, _vp, _vp, i32, i32, P(SummaryDesc), _vp],
        "eta_predict_threshold": [i32, i32, i32, i32, _vp, _vp, _vp, _vp, _vp],
        "eta_decode_workspace_size": [P(KvDesc), ctypes.c_int64, P(DecodeParams), P(sz)],
        "eta_decode": [P(KvDesc), i32, _vp, _vp, _vp, _vp, P(SummaryDesc), _vp, P(DecodeParams),
                       _vp, _vp, _vp, _vp, _vp, sz, _vp],
        "eta_decode_predicted": [P(KvDesc), i32, _vp, _vp, _vp, _vp, P(SummaryDesc), _vp, _vp,
                                 P(DecodeParams), _vp, _vp, _vp, _vp, _vp, _vp, sz, _vp],
        "eta_decode_predicted_noalloc": [P(KvDesc), i32, _vp, _vp, _vp, _vp, P(SummaryDesc), _vp,
                                         _vp, P(DecodeParams), _vp, _vp, _vp, _vp, _vp, _vp],
        "eta_block_bounds": [P(KvDesc), i32, _vp, _vp, P(SummaryDesc), f32, _vp, _vp],
        "eta_dense_workspace_size": [P(KvDesc), i32, P(sz)],
        "eta_dense_decode": [P(KvDesc), i32, _vp, _vp, _vp, _vp, _vp, i32, _vp, sz, _vp],
        "eta_profile_begin": [],
        "eta_profile_end": [P(KernelTime)],
    }
    for name, args in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.eta_last_error_string.restype = ctypes.c_char_p
    lib.eta_last_error_string.argtypes = []
    lib.eta_abi_version.restype = ctypes.c_int32
    if path is None:
        _lib = lib
    return lib


def _check(status: int):
    if status != ETA_OK:
        raise EtaError(status, load_library().eta_last_error_string().decode())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return ETA_DT_F32
    if t.dtype == torch.bfloat16:
        return ETA_DT_BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else _vp(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return _vp(s.cuda_stream)


# ---------------------------------------------------------------- descriptors

def kv_desc(k: torch.Tensor, num_q_heads: int, block_size: int) -> KvDesc:
    """Descriptor of a [B][Hkv][T_cap][d] cache (any strides, head dim contiguous)."""
    if k.dim() != 4 or k.stride(3) != 1:
        raise ValueError("K/V must be 4-D [B][Hkv][T_cap][d] with a contiguous head dimension")
    B, Hkv, T_cap, d = k.shape
    return KvDesc(batch=B, num_q_heads=num_q_heads, num_kv_heads=Hkv, head_dim=d,
                  block_size=block_size, kv_dtype=_dtype_code(k), capacity_tokens=T_cap,
                  stride_b=k.stride(0), stride_h=k.stride(1), stride_t=k.stride(2))


@dataclass
class Summaries:
    """Block index: mu, sigma [B][Hkv][d][n_blk_cap] (dimension-major), max_norm [B][Hkv][n_blk_cap]."""
    mu: torch.Tensor
    sigma: torch.Tensor
    max_norm: torch.Tensor

    @property
    def n_blk_cap(self) -> int:
        return self.mu.shape[-1]

    def desc(self) -> SummaryDesc:
        st = {torch.float32: ETA_DT_F32, torch.float16: ETA_DT_F16,
              torch.float8_e4m3fn: ETA_DT_FP8}[self.mu.dtype]
        return SummaryDesc(mu=_ptr(self.mu), sigma=_ptr(self.sigma), max_norm=_ptr(self.max_norm),
                           n_blk_cap=self.n_blk_cap, stat_dtype=st)

    @staticmethod
    def empty(B: int, Hkv: int, d: int, n_blk_cap: int, device,
              stat_dtype: torch.dtype = torch.float32) -> "Summaries":
        """stat_dtype: torch.float32, torch.float16 or torch.float8_e4m3fn (mu and sigma
        records; FP8 as 8-bit E4M3 codes, nearest even, saturating at +-448)."""
        n = max(int(n_blk_cap), 1)
        if stat_dtype not in (torch.float32, torch.float16, torch.float8_e4m3fn):
            raise TypeError(f"unsupported record dtype {stat_dtype}")

        def rec():   # zero bits (zero in all three formats), filled as plain words
            if stat_dtype == torch.float8_e4m3fn:
                return torch.zeros(B, Hkv, d, n, device=device, dtype=torch.uint8).view(stat_dtype)
            return torch.zeros(B, Hkv, d, n, device=device, dtype=stat_dtype)
        return Summaries(mu=rec(), sigma=rec(),
                         max_norm=torch.zeros(B, Hkv, n, device=device, dtype=torch.float32))


def decode_params(*, beta=4.0, z=1.0, offset_a=0.0, rescue_window=128, lwb=0,
                  self_ungated=False, screen_all=False, num_splits=0) -> DecodeParams:
    return DecodeParams(beta=beta, z=z, offset_a=offset_a, rescue_window_blocks=rescue_window,
                        pin_recent_blocks=lwb, self_ungated=int(bool(self_ungated)),
                        screen_all=int(bool(screen_all)), num_splits=num_splits)


# ---------------------------------------------------------------- entry points

def build_block_summaries(k: torch.Tensor, seq_lens: torch.Tensor, block_size: int, *,
                          num_q_heads: Optional[int] = None, out: Optional[Summaries] = None,
                          sub_block: int = 0, stat_dtype: torch.dtype = torch.float32,
                          stream=None) -> Summaries:
    """eta_build_block_summaries: mu, sigma, M of every full block of K
    (sub_block > 0: eta_build_block_summaries_envelope, sigma = sub-block envelope;
    stat_dtype torch.float16 / torch.float8_e4m3fn: half-precision / FP8 E4M3 mu / sigma
    records)."""
    B, Hkv, T_cap, d = k.shape
    desc = kv_desc(k, num_q_heads or Hkv, block_size)
    if out is None:
        out = Summaries.empty(B, Hkv, d, T_cap // block_size, k.device, stat_dtype)
    sd = out.desc()
    lib = load_library()
    if sub_block:
        _check(lib.eta_build_block_summaries_envelope(ctypes.byref(desc), _ptr(k), _ptr(seq_lens),
                                                      sub_block, ctypes.byref(sd), _stream(stream)))
    else:
        _check(lib.eta_build_block_summaries(ctypes.byref(desc), _ptr(k), _ptr(seq_lens),
                                             ctypes.byref(sd), _stream(stream)))
    return out


def update_block_summaries(k: torch.Tensor, prev_lens: torch.Tensor, seq_lens: torch.Tensor,
                           summ: Summaries, block_size: int, *, max_new_blocks: int = 1,
                           num_q_heads: Optional[int] = None, sub_block: int = 0,
                           stream=None) -> Summaries:
    """eta_update_block_summaries: records of the blocks completed since prev_lens."""
    desc = kv_desc(k, num_q_heads or k.shape[1], block_size)
    sd = summ.desc()
    _check(load_library().eta_update_block_summaries(ctypes.byref(desc), _ptr(k), _ptr(prev_lens),
                                                     _ptr(seq_lens), max_new_blocks, sub_block,
                                                     ctypes.byref(sd), _stream(stream)))
    return summ


def _check_predictor(q: torch.Tensor, W: Optional[torch.Tensor], bias: torch.Tensor) -> None:
    """The predictor's tensors as the C ABI reads them (it sees only pointers): q
    contiguous [B][Hq][d]; W None or fp32 [Hq][Hq d] contiguous (head-major); bias
    fp32 [Hq] contiguous."""
    B, Hq, d = q.shape
    if not q.is_contiguous():
        raise ValueError("q must be contiguous [B][Hq][d]")
    if W is not None and (W.dtype != torch.float32 or tuple(W.shape) != (Hq, Hq * d)
                          or not W.is_contiguous()):
        raise ValueError(f"W must be fp32 [{Hq}][{Hq * d}] contiguous (head-major: row h holds "
                         f"head h's weights), got {W.dtype} {tuple(W.shape)}")
    if bias.dtype != torch.float32 or tuple(bias.shape) != (Hq,) or not bias.is_contiguous():
        raise ValueError(f"bias must be fp32 [{Hq}] contiguous, got {bias.dtype} {tuple(bias.shape)}")


def predict_threshold(q: torch.Tensor, W: Optional[torch.Tensor], bias: torch.Tensor, *,
                      out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """eta_predict_threshold: tau[b][h] = concat(q[b]) . W[h] + bias[h] (W None: tau = bias).
    W is head-major, fp32 [Hq][Hq d]: row h holds the weights of head h's threshold
    (the (Hq d) x Hq predictor matrix transposed)."""
    B, Hq, d = q.shape
    _check_predictor(q, W, bias)
    if out is None:
        out = torch.empty(B, Hq, device=q.device, dtype=torch.float32)
    _check(load_library().eta_predict_threshold(B, Hq, d, _dtype_code(q), _ptr(q), _ptr(W),
                                                _ptr(bias), _ptr(out), _stream(stream)))
    return out


def decode_workspace_size(desc: KvDesc, n_blk_cap: int, params: DecodeParams) -> int:
    """eta_decode_workspace_size for a summary of block capacity n_blk_cap."""
    n = ctypes.c_size_t()
    _check(load_library().eta_decode_workspace_size(ctypes.byref(desc), int(n_blk_cap),
                                                    ctypes.byref(params), ctypes.byref(n)))
    return n.value


def alloc_workspace(nbytes: int, device) -> torch.Tensor:
    """Workspace buffer (torch's caching allocator returns 256-byte aligned blocks)."""
    t = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    assert t.data_ptr() % 256 == 0
    return t


@dataclass
class DecodeOut:
    out: torch.Tensor            # [B][Hq][d], dtype of q
    mask: torch.Tensor           # [B][Hq][n_blk_cap] uint8
    counts: Optional[torch.Tensor]  # [B][Hq] int32
    union_counts: Optional[torch.Tensor] = None  # [B][Hkv] int32 GQA union blocks


def _decode_outputs(q, k, summ, out, mask, counts, union_counts, want_counts):
    B, Hq, _ = q.shape
    if out is None:
        out = torch.empty_like(q)
    if mask is None:
        mask = torch.empty(B, Hq, summ.n_blk_cap, dtype=torch.uint8, device=q.device)
    if counts is None and want_counts:
        counts = torch.empty(B, Hq, dtype=torch.int32, device=q.device)
    if union_counts is None and want_counts:
        union_counts = torch.empty(B, k.shape[1], dtype=torch.int32, device=q.device)
    return out, mask, counts, union_counts


def decode(q, k, v, seq_lens, summ: Summaries, tau, *, block_size: int,
           params: Optional[DecodeParams] = None, out=None, mask=None, counts=None,
           union_counts=None, want_counts: bool = True,
           workspace: Optional[torch.Tensor] = None, stream=None) -> DecodeOut:
    """eta_decode: one ETA decode step -> output, selected-block mask, attended token
    counts per head and GQA union counts per (sequence, kv head)."""
    B, Hq, d = q.shape
    p = params if params is not None else decode_params()
    desc = kv_desc(k, Hq, block_size)
    if v.shape != k.shape or v.stride() != k.stride() or v.dtype != k.dtype:
        raise ValueError("K and V must share shape, strides and dtype")
    out, mask, counts, union_counts = _decode_outputs(q, k, summ, out, mask, counts, union_counts,
                                                      want_counts)
    nbytes = decode_workspace_size(desc, summ.n_blk_cap, p)
    if workspace is None or workspace.numel() < nbytes:
        workspace = alloc_workspace(nbytes, q.device)
    sd = summ.desc()
    _check(load_library().eta_decode(ctypes.byref(desc), _dtype_code(q), _ptr(q), _ptr(k), _ptr(v),
                                     _ptr(seq_lens), ctypes.byref(sd), _ptr(tau), ctypes.byref(p),
                                     _ptr(out), _ptr(mask), _ptr(counts), _ptr(union_counts),
                                     _ptr(workspace), workspace.numel(), _stream(stream)))
    return DecodeOut(out=out, mask=mask, counts=counts, union_counts=union_counts)


def decode_predicted(q, k, v, seq_lens, summ: Summaries, W, bias, *, block_size: int,
                     params: Optional[DecodeParams] = None, out=None, mask=None, counts=None,
                     union_counts=None, tau_out=None, want_counts: bool = True,
                     workspace: Optional[torch.Tensor] = None, stream=None) -> DecodeOut:
    """eta_decode_predicted: predictor fused into the decode step (tau as in
    predict_threshold, W head-major)."""
    B, Hq, d = q.shape
    _check_predictor(q, W, bias)
    p = params if params is not None else decode_params()
    desc = kv_desc(k, Hq, block_size)
    if v.shape != k.shape or v.stride() != k.stride() or v.dtype != k.dtype:
        raise ValueError("K and V must share shape, strides and dtype")
    out, mask, counts, union_counts = _decode_outputs(q, k, summ, out, mask, counts, union_counts,
                                                      want_counts)
    nbytes = decode_workspace_size(desc, summ.n_blk_cap, p)
    if workspace is None or workspace.numel() < nbytes:
        workspace = alloc_workspace(nbytes, q.device)
    sd = summ.desc()
    _check(load_library().eta_decode_predicted(
        ctypes.byref(desc), _dtype_code(q), _ptr(q), _ptr(k), _ptr(v), _ptr(seq_lens),
        ctypes.byref(sd), _ptr(W), _ptr(bias), ctypes.byref(p), _ptr(out), _ptr(mask),
        _ptr(counts), _ptr(union_counts), _ptr(tau_out), _ptr(workspace), workspace.numel(),
        _stream(stream)))
    return DecodeOut(out=out, mask=mask, counts=counts, union_counts=union_counts)


NOALLOC_SCRATCH_BYTES = 32 << 20   # ETA_DECODE_NOALLOC_SCRATCH_BYTES


def decode_predicted_noalloc(q, k, v, seq_lens, summ: Summaries, W, bias, *, block_size: int,
                             params: Optional[DecodeParams] = None, out=None, mask=None,
                             counts=None, union_counts=None, tau_out=None,
                             want_counts: bool = True, stream=None) -> DecodeOut:
    """eta_decode_predicted_noalloc: eta_decode_predicted with the library's own scratch
    as the workspace (the C call allocates nothing; output buffers not given are
    allocated here, before the call)."""
    B, Hq, d = q.shape
    _check_predictor(q, W, bias)
    p = params if params is not None else decode_params()
    desc = kv_desc(k, Hq, block_size)
    if v.shape != k.shape or v.stride() != k.stride() or v.dtype != k.dtype:
        raise ValueError("K and V must share shape, strides and dtype")
    out, mask, counts, union_counts = _decode_outputs(q, k, summ, out, mask, counts, union_counts,
                                                      want_counts)
    sd = summ.desc()
    _check(load_library().eta_decode_predicted_noalloc(
        ctypes.byref(desc), _dtype_code(q), _ptr(q), _ptr(k), _ptr(v), _ptr(seq_lens),
        ctypes.byref(sd), _ptr(W), _ptr(bias), ctypes.byref(p), _ptr(out), _ptr(mask),
        _ptr(counts), _ptr(union_counts), _ptr(tau_out), _stream(stream)))
    return DecodeOut(out=out, mask=mask, counts=counts, union_counts=union_counts)


class DecodeStep:
    """A prepared eta_decode_predicted call: descriptors, parameters, output
    buffers and the workspace are set up once; ``run()`` is a single C call
    with cached arguments (what a serving loop would do every token).  The
    thresholds are read from ``bias`` (and W) at every call, so updating those
    tensors in place takes effect on the next step."""

    def __init__(self, q, k, v, seq_lens, summ: Summaries, W, bias, *, block_size: int,
                 params: Optional[DecodeParams] = None, want_counts: bool = True, stream=None):
        B, Hq, d = q.shape
        _check_predictor(q, W, bias)
        self.tensors = (q, k, v, seq_lens, summ.mu, summ.sigma, summ.max_norm, W, bias)
        self.params = params if params is not None else decode_params()
        self.desc = kv_desc(k, Hq, block_size)
        self.sdesc = summ.desc()
        self.out = torch.empty_like(q)
        self.mask = torch.empty(B, Hq, summ.n_blk_cap, dtype=torch.uint8, device=q.device)
        self.counts = torch.empty(B, Hq, dtype=torch.int32, device=q.device) if want_counts else None
        self.union_counts = (torch.empty(B, k.shape[1], dtype=torch.int32, device=q.device)
                             if want_counts else None)
        self.tau = torch.empty(B, Hq, dtype=torch.float32, device=q.device)
        self.workspace = alloc_workspace(decode_workspace_size(self.desc, summ.n_blk_cap, self.params),
                                         q.device)
        self._fn = load_library().eta_decode_predicted
        self._args = (ctypes.byref(self.desc), _dtype_code(q), _ptr(q), _ptr(k), _ptr(v),
                      _ptr(seq_lens), ctypes.byref(self.sdesc), _ptr(W), _ptr(bias),
                      ctypes.byref(self.params), _ptr(self.out), _ptr(self.mask),
                      _ptr(self.counts), _ptr(self.union_counts), _ptr(self.tau),
                      _ptr(self.workspace), self.workspace.numel(), _stream(stream))

    def run(self) -> None:
        st = self._fn(*self._args)
        if st != ETA_OK:
            _check(st)


def block_bounds(q, seq_lens, summ: Summaries, k_like: torch.Tensor, *, block_size: int,
                 z: float, out=None, stream=None) -> torch.Tensor:
    """eta_block_bounds: the screening bound of every full block and query head (NaN beyond N_b)."""
    B, Hq, d = q.shape
    desc = kv_desc(k_like, Hq, block_size)
    if out is None:
        out = torch.empty(B, Hq, summ.n_blk_cap, dtype=torch.float32, device=q.device)
    sd = summ.desc()
    _check(load_library().eta_block_bounds(ctypes.byref(desc), _dtype_code(q), _ptr(q),
                                           _ptr(seq_lens), ctypes.byref(sd), ctypes.c_float(z),
                                           _ptr(out), _stream(stream)))
    return out


def dense_workspace_size(desc: KvDesc, num_splits: int = 0) -> int:
    n = ctypes.c_size_t()
    _check(load_library().eta_dense_workspace_size(ctypes.byref(desc), num_splits, ctypes.byref(n)))
    return n.value


def dense_decode(q, k, v, seq_lens, *, block_size: int = 64, num_splits: int = 0, out=None,
                 workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """eta_dense_decode: plain softmax attention over every token (the dense baseline)."""
    B, Hq, d = q.shape
    desc = kv_desc(k, Hq, block_size)
    if out is None:
        out = torch.empty_like(q)
    nbytes = dense_workspace_size(desc, num_splits)
    if workspace is None or workspace.numel() < nbytes:
        workspace = alloc_workspace(nbytes, q.device)
    _check(load_library().eta_dense_decode(ctypes.byref(desc), _dtype_code(q), _ptr(q), _ptr(k),
                                           _ptr(v), _ptr(seq_lens), _ptr(out), num_splits,
                                           _ptr(workspace), workspace.numel(), _stream(stream)))
    return out


def profile_begin():
    _check(load_library().eta_profile_begin())


def profile_end() -> dict:
    arr = (KernelTime * len(KERNEL_KINDS))()
    _check(load_library().eta_profile_end(arr))
    return {name: (arr[i].ms_total, arr[i].launches) for i, name in enumerate(KERNEL_KINDS)}


CALIB_UNIT = float(2 ** 40)   # fixed-point unit of the calibration accumulators


class Calibrator:
    """Offline density-matched calibration of static per-head thresholds
    (eta_calib_accumulate / eta_calib_solve).  The accumulators live on the
    device; ``accumulate`` may be called for any number of batches of
    calibration sequences, ``solve`` returns the constants (usable as the
    ``bias`` of a predictor-free decode, W = None)."""

    def __init__(self, num_q_heads: int, num_kv_heads: int, head_dim: int, *, beta: float,
                 lo: float, hi: float, num_bins: int, device):
        self.Hq, self.Hkv, self.d = num_q_heads, num_kv_heads, head_dim
        self.beta, self.lo, self.hi, self.nb = float(beta), float(lo), float(hi), int(num_bins)
        self.hist = torch.zeros(num_q_heads, num_bins, dtype=torch.int64, device=device)
        self.density = torch.zeros(num_q_heads, dtype=torch.int64, device=device)

    def _desc(self, N: int, T: int) -> CalibDesc:
        return CalibDesc(num_seqs=N, num_q_heads=self.Hq, num_kv_heads=self.Hkv, head_dim=self.d,
                         seq_len=T, dtype=ETA_DT_BF16, beta=self.beta, lo=self.lo, hi=self.hi,
                         num_bins=self.nb)

    def _state(self) -> CalibState:
        return CalibState(hist=_ptr(self.hist), density=_ptr(self.density))

    def accumulate(self, q: torch.Tensor, k: torch.Tensor, tau: torch.Tensor, stream=None):
        """q bf16 [N][Hq][T][d], k bf16 [N][Hkv][T][d], tau fp32 [N][Hq][T] (contiguous)."""
        N, Hq, T, d = q.shape
        assert (Hq, d) == (self.Hq, self.d) and k.shape == (N, self.Hkv, T, d)
        assert tau.shape == (N, Hq, T) and tau.dtype == torch.float32
        assert q.is_contiguous() and k.is_contiguous() and tau.is_contiguous()
        desc, st = self._desc(N, T), self._state()
        _check(load_library().eta_calib_accumulate(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(tau),
                                                   ctypes.byref(st), _stream(stream)))

    def solve(self, stream=None):
        """(c fp32 [Hq], target density fp64 [Hq])."""
        c = torch.empty(self.Hq, dtype=torch.float32, device=self.hist.device)
        target = torch.empty(self.Hq, dtype=torch.float64, device=self.hist.device)
        desc, st = self._desc(1, 1), self._state()
        _check(load_library().eta_calib_solve(ctypes.byref(desc), ctypes.byref(st), _ptr(c),
                                              _ptr(target), _stream(stream)))
        return c, target


def gated_prefill(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, tau: torch.Tensor,
                  seq_lens: torch.Tensor, *, beta: float, additive: bool = False, C: float = 0.0,
                  out: Optional[torch.Tensor] = None, R: Optional[torch.Tensor] = None,
                  L: Optional[torch.Tensor] = None, stream=None):
    """eta_gated_prefill: gated causal attention forward with the gate row sums R and
    the log-sum-exp L.  q bf16 [B][Hq][T][d], k, v bf16 [B][Hkv][T][d], tau fp32
    [B][Hq][T], seq_lens int32 [B]; returns (out bf16 [B][Hq][T][d], R, L fp32 [B][Hq][T])."""
    B, Hq, T, d = q.shape
    Hkv = k.shape[1]
    assert k.shape == (B, Hkv, T, d) and v.shape == k.shape and tau.shape == (B, Hq, T)
    assert q.dtype == k.dtype == v.dtype == torch.bfloat16 and tau.dtype == torch.float32
    assert q.is_contiguous() and k.is_contiguous() and v.is_contiguous() and tau.is_contiguous()
    if out is None:
        out = torch.empty_like(q)
    if R is None:
        R = torch.empty(B, Hq, T, dtype=torch.float32, device=q.device)
    if L is None:
        L = torch.empty(B, Hq, T, dtype=torch.float32, device=q.device)
    desc = PrefillDesc(batch=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, capacity_tokens=T,
                       dtype=ETA_DT_BF16, beta=beta, additive=int(bool(additive)), C=C)
    _check(load_library().eta_gated_prefill(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v),
                                            _ptr(tau), _ptr(seq_lens), _ptr(out), _ptr(R), _ptr(L),
                                            _stream(stream)))
    return out, R, L
