"""fp64 CPU oracle of the ETA decode path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never uses it.

Inputs are numpy arrays: ``float32`` for fp32 data, ``uint16`` for bf16 data
given as raw 16-bit words (upcast exactly inside the C code).  All arithmetic
is double precision (``eta_oracle.c``).  What each function follows in the
paper is stated in the C source and repeated briefly below.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# ETA_ORACLE_LIB lets the mutation test point the wrapper at a deliberately broken build.
_LIB_PATH = os.environ.get("ETA_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

F32, BF16 = 0, 1

_dp = ctypes.POINTER(ctypes.c_double)
_vp = ctypes.c_void_p


class _Problem(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int32), ("Hq", ctypes.c_int32), ("Hkv", ctypes.c_int32),
        ("d", ctypes.c_int32), ("b", ctypes.c_int32),
        ("T_cap", ctypes.c_int64),
        ("q_dtype", ctypes.c_int32), ("kv_dtype", ctypes.c_int32),
        ("q", _vp), ("k", _vp), ("v", _vp),
        ("seq_lens", _vp), ("tau", _vp),
        ("beta", ctypes.c_double), ("z", ctypes.c_double), ("a", ctypes.c_double),
        ("c", ctypes.c_int32), ("lwb", ctypes.c_int32), ("self_ungated", ctypes.c_int32),
        ("screen_all", ctypes.c_int32), ("gate_off", ctypes.c_int32),
        ("bounds_only", ctypes.c_int32),
        ("mu", _vp), ("sigma", _vp), ("maxnorm", _vp),
        ("sel_in", _vp),
        ("rows", _vp), ("n_rows", ctypes.c_int32),
        ("n_threads", ctypes.c_int32),
        ("o", _vp), ("sel", _vp), ("bounds", _vp), ("counts", _vp), ("lse", _vp),
        ("rescued", _vp),
        ("blockmax", _vp), ("quality", _vp), ("missed", _vp),
    ]


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.eta_oracle_gate.restype = ctypes.c_double
    lib.eta_oracle_gate.argtypes = [ctypes.c_double] * 3
    lib.eta_oracle_summaries.restype = None
    lib.eta_oracle_summaries.argtypes = [_vp, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                                         ctypes.c_int, ctypes.c_int, _vp, _vp, _vp]
    lib.eta_oracle_envelope.restype = None
    lib.eta_oracle_envelope.argtypes = [_vp, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                                        ctypes.c_int, ctypes.c_int, ctypes.c_int, _vp, _vp]
    lib.eta_oracle_calib_hist.restype = None
    lib.eta_oracle_calib_hist.argtypes = [_vp, _vp, ctypes.c_int, _vp, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                          ctypes.c_double, ctypes.c_double, ctypes.c_int,
                                          ctypes.c_double, ctypes.c_double, _vp, _vp, _vp, _vp, _vp]
    lib.eta_oracle_calib_g.restype = ctypes.c_double
    lib.eta_oracle_calib_g.argtypes = [_vp, ctypes.c_int, ctypes.c_double, ctypes.c_double,
                                       ctypes.c_double, ctypes.c_double]
    lib.eta_oracle_calib_solve.restype = ctypes.c_double
    lib.eta_oracle_calib_solve.argtypes = [_vp, ctypes.c_int, ctypes.c_double, ctypes.c_double,
                                           ctypes.c_double, ctypes.c_double]
    lib.eta_oracle_prefill.restype = None
    lib.eta_oracle_prefill.argtypes = [_vp, _vp, _vp, ctypes.c_int, _vp, _vp, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_double, ctypes.c_int, ctypes.c_double, _vp, _vp, _vp]
    lib.eta_oracle_prefill_rows.restype = None
    lib.eta_oracle_prefill_rows.argtypes = [_vp, _vp, _vp, ctypes.c_int, _vp, _vp, ctypes.c_int,
                                            ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                            ctypes.c_double, ctypes.c_int, ctypes.c_double, _vp,
                                            ctypes.c_int, _vp, _vp, _vp]
    lib.eta_oracle_round_f16.restype = ctypes.c_double
    lib.eta_oracle_round_f16.argtypes = [ctypes.c_double]
    lib.eta_oracle_round_f16_array.restype = None
    lib.eta_oracle_round_f16_array.argtypes = [_vp, _vp, ctypes.c_int64]
    lib.eta_oracle_round_e4m3_array.restype = None
    lib.eta_oracle_round_e4m3_array.argtypes = [_vp, _vp, ctypes.c_int64]
    lib.eta_oracle_bound.restype = ctypes.c_double
    lib.eta_oracle_bound.argtypes = [_vp, _vp, _vp, ctypes.c_double, ctypes.c_int, ctypes.c_double]
    lib.eta_oracle_predict.restype = None
    lib.eta_oracle_predict.argtypes = [_vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_int, _vp, _vp, _vp]
    lib.eta_oracle_select.restype = ctypes.c_int64
    lib.eta_oracle_select.argtypes = [_vp, ctypes.c_int64, ctypes.c_double, ctypes.c_int,
                                      ctypes.c_int, ctypes.c_int, _vp]
    lib.eta_oracle_attend.restype = None
    lib.eta_oracle_attend.argtypes = [_vp, _vp, _vp, ctypes.c_int, ctypes.c_int64,
                                      ctypes.c_int64, ctypes.c_int, ctypes.c_int, _vp,
                                      ctypes.c_int, ctypes.c_double, ctypes.c_double,
                                      ctypes.c_int, ctypes.c_int, _vp, _vp, _vp]
    lib.eta_oracle_screen_quality.restype = None
    lib.eta_oracle_screen_quality.argtypes = [_vp, _vp, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                                              ctypes.c_int, ctypes.c_int, _vp, ctypes.c_double,
                                              ctypes.c_double, ctypes.c_int, ctypes.c_int, _vp,
                                              _vp, _vp]
    lib.eta_oracle_decode.restype = ctypes.c_int
    lib.eta_oracle_decode.argtypes = [ctypes.POINTER(_Problem)]
    _lib = lib
    return lib


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError(f"oracle takes float32 or uint16 (bf16 bits) arrays, got {a.dtype}")


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(_vp)


def _c(a, dtype=None):
    if a is None:
        return None
    a = np.asarray(a) if dtype is None else np.asarray(a, dtype=dtype)
    return np.ascontiguousarray(a)


# ------------------------------------------------------------------ pieces

def gate(S: float, tau: float, beta: float) -> float:
    """Gated score S * sigmoid(beta (S - tau)) -- Eq. (soft_mask) x Eq. (mult_attn)."""
    return _load().eta_oracle_gate(float(S), float(tau), float(beta))


def summaries(k: np.ndarray, b: int):
    """(mu, sigma, M) of the full blocks of one key sequence ``k[T][d]``.

    Population mean / standard deviation per coordinate and the largest key
    norm, Sec. "Block-Based Scanning via Dual Metadata Caching".
    """
    k = _c(k)
    T, d = k.shape
    N = T // b
    mu = np.zeros((max(N, 1), d)); sg = np.zeros((max(N, 1), d)); mx = np.zeros(max(N, 1))
    _load().eta_oracle_summaries(_ptr(k), _dtype_code(k), d, T, d, b, _ptr(mu), _ptr(sg), _ptr(mx))
    return mu[:N], sg[:N], mx[:N]


def round_f16(x) -> np.ndarray:
    """Nearest binary16 values (ties to even) as float64: the fp16 index records of
    App. "GQA-Grouped Execution and Compact Metadata Layout"."""
    a = np.ascontiguousarray(np.asarray(x, np.float64))
    out = np.empty_like(a)
    _load().eta_oracle_round_f16_array(_ptr(a), _ptr(out), a.size)
    return out


def round_e4m3(x) -> np.ndarray:
    """Nearest 8-bit E4M3 values (ties to even, saturating at +-448) as float64: the
    FP8 index records (Sec. "Limitations and Conclusion": FP8 metadata quantisation)."""
    a = np.ascontiguousarray(np.asarray(x, np.float64))
    out = np.empty_like(a)
    _load().eta_oracle_round_e4m3_array(_ptr(a), _ptr(out), a.size)
    return out


def envelope(k: np.ndarray, b: int, b_sub: int, mu: np.ndarray) -> np.ndarray:
    """Sub-block envelope standard deviation, Eq. (subblock_envelope_appx)."""
    k = _c(k)
    T, d = k.shape
    N = T // b
    env = np.zeros((max(N, 1), d))
    mu = _c(mu, np.float64)
    _load().eta_oracle_envelope(_ptr(k), _dtype_code(k), d, T, d, b, b_sub, _ptr(mu), _ptr(env))
    return env[:N]


def bound(q: np.ndarray, mu: np.ndarray, sigma: np.ndarray, M: float, z: float) -> float:
    """Score_dual(q, B), Eq. (dual_bound_eq), for one head and one block."""
    q = _c(q, np.float64); mu = _c(mu, np.float64); sigma = _c(sigma, np.float64)
    return _load().eta_oracle_bound(_ptr(q), _ptr(mu), _ptr(sigma), float(M), q.shape[0], float(z))


def predict(q: np.ndarray, W: Optional[np.ndarray], bias: Optional[np.ndarray]) -> np.ndarray:
    """tau[B][Hq] = concat_h(q[b,h,:]) W + bias, Eq. (tau_pred); W None -> bias."""
    q = _c(q)
    B, Hq, d = q.shape
    W = _c(W, np.float32)
    bias = _c(bias, np.float32)
    tau = np.zeros((B, Hq))
    _load().eta_oracle_predict(_ptr(q), _dtype_code(q), B, Hq, d, _ptr(W), _ptr(bias), _ptr(tau))
    return tau


def select(bounds: np.ndarray, tau_eff: float, c: int, lwb: int = 0, screen_all: bool = False):
    """Selection with pins and top-1 rescue for one head -> (sel uint8[N], rescued index or -1)."""
    bounds = _c(bounds, np.float64)
    N = bounds.shape[0]
    sel = np.zeros(max(N, 1), np.uint8)
    r = _load().eta_oracle_select(_ptr(bounds), N, float(tau_eff), int(c), int(lwb),
                                  int(bool(screen_all)), _ptr(sel))
    return sel[:N], int(r)


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, b: int, sel: np.ndarray, *,
           use_tail: bool = True, tau_eff: float = float("-inf"), beta: float = 4.0,
           self_ungated: bool = False, gate_off: bool = False):
    """Gated softmax attention of one head over selected blocks (+ tail) -> (o, lse, count)."""
    q = _c(q, np.float64); k = _c(k); v = _c(v)
    T, d = k.shape
    assert v.shape == k.shape and v.dtype == k.dtype
    N = T // b
    sel = np.ascontiguousarray(np.asarray(sel, np.uint8).reshape(-1)[:N])
    if sel.shape[0] < 1:
        sel = np.zeros(1, np.uint8)
    o = np.zeros(d); lse = ctypes.c_double(); cnt = ctypes.c_int64()
    _load().eta_oracle_attend(_ptr(q), _ptr(k), _ptr(v), _dtype_code(k), d, T, d, b, _ptr(sel),
                              int(use_tail), float(tau_eff), float(beta), int(self_ungated),
                              int(gate_off), _ptr(o), ctypes.byref(lse), ctypes.byref(cnt))
    return o, lse.value, cnt.value


QUALITY_FIELDS = ("positive_blocks", "false_negative_blocks", "false_positive_blocks",
                  "selected_blocks", "above_keys", "above_keys_attended")


def screen_quality(q: np.ndarray, k: np.ndarray, b: int, sel: np.ndarray, *, tau_eff: float,
                   beta: float = 4.0, self_ungated: bool = False, gate_off: bool = False) -> dict:
    """Screening-quality diagnostics of one head over keys ``k[T][d]`` and a block
    selection ``sel[N]`` (Tab. "index_quality"): brute-force block maxima, positive /
    false-negative / false-positive / selected blocks, above-threshold keys of the full
    blocks and how many are attended, and the missed gated softmax mass of the
    rejected blocks (see eta_oracle_screen_quality)."""
    q = _c(q, np.float64); k = _c(k)
    T, d = k.shape
    N = T // b
    s = np.zeros(max(N, 1), np.uint8)
    s[:N] = np.asarray(sel, np.uint8).reshape(-1)[:N]
    bm = np.full(max(N, 1), np.nan)
    qual = np.zeros(6, np.int64)
    missed = ctypes.c_double()
    _load().eta_oracle_screen_quality(_ptr(q), _ptr(k), _dtype_code(k), d, T, d, b, _ptr(s),
                                      float(tau_eff), float(beta), int(self_ungated),
                                      int(gate_off), _ptr(bm), _ptr(qual), ctypes.byref(missed))
    out = dict(zip(QUALITY_FIELDS, (int(x) for x in qual)))
    out["blockmax"] = bm[:N]
    out["missed_mass"] = missed.value
    return out


def quality_rates(res: "DecodeResult", rows: Optional[Sequence[int]] = None) -> dict:
    """Pooled screening-quality rates of a decode run with ``quality=True``:
    block false-negative rate (false negatives / positive blocks), false-positive
    rate (selected blocks that are not positive / selected blocks), token recall
    (attended above-threshold keys / above-threshold keys) and the missed gated
    mass (mean over rows and largest row)."""
    B, Hq = res.missed.shape
    rows = list(range(B * Hq)) if rows is None else list(rows)
    qs = np.array([res.quality[r // Hq, r % Hq] for r in rows], np.int64).reshape(-1, 6)
    mm = np.array([res.missed[r // Hq, r % Hq] for r in rows])
    tot = qs.sum(axis=0)
    ratio = lambda a, b: float(a) / float(b) if b else None
    return {"rows": len(rows), "positive_blocks": int(tot[0]),
            "false_negative_rate": ratio(tot[1], tot[0]), "false_positive_rate": ratio(tot[2], tot[3]),
            "token_recall": ratio(tot[5], tot[4]), "missed_mass_mean": float(mm.mean()) if mm.size else None,
            "missed_mass_max": float(mm.max()) if mm.size else None,
            "rows_with_false_negatives": int(np.count_nonzero(qs[:, 1]))}


# ------------------------------------------------------------------ batched

@dataclass
class DecodeResult:
    o: np.ndarray          # [B][Hq][d] float64
    sel: np.ndarray        # [B][Hq][N_cap] uint8
    bounds: np.ndarray     # [B][Hq][N_cap] float64 (NaN beyond N_b)
    counts: np.ndarray     # [B][Hq] int64
    lse: np.ndarray        # [B][Hq] float64
    rescued: np.ndarray    # [B][Hq] int64 (-1: no rescue)
    blockmax: Optional[np.ndarray] = None   # [B][Hq][N_cap] (quality=True; NaN beyond N_b)
    quality: Optional[np.ndarray] = None    # [B][Hq][6] QUALITY_FIELDS (quality=True)
    missed: Optional[np.ndarray] = None     # [B][Hq] missed gated mass (quality=True)


def block_index(k: np.ndarray, seq_lens: Sequence[int], block_size: int, n_threads: int = 0):
    """Summaries (mu, sigma, M) of every full block of every (sequence, kv head).

    k [B][Hkv][T_cap][d] -> mu, sigma [B][Hkv][N_cap][d] and M [B][Hkv][N_cap] (float64),
    zero for blocks that are not full.  Same arithmetic as ``summaries``.
    """
    import concurrent.futures as cf
    k = _c(k)
    B, Hkv, T_cap, d = k.shape
    Ncap = T_cap // block_size
    mu = np.zeros((B, Hkv, max(Ncap, 1), d)); sg = np.zeros_like(mu)
    mx = np.zeros((B, Hkv, max(Ncap, 1)))
    lib = _load()
    code = _dtype_code(k)

    def one(bg):
        b, g = divmod(bg, Hkv)
        T = max(0, min(int(seq_lens[b]), T_cap))
        sub = k[b, g]
        lib.eta_oracle_summaries(_ptr(sub), code, d, T, d, block_size,
                                 mu[b, g].ctypes.data_as(_vp), sg[b, g].ctypes.data_as(_vp),
                                 mx[b, g].ctypes.data_as(_vp))
    workers = n_threads if n_threads > 0 else (os.cpu_count() or 1)
    with cf.ThreadPoolExecutor(max_workers=workers) as ex:   # ctypes releases the GIL
        list(ex.map(one, range(B * Hkv)))
    return mu[:, :, :Ncap], sg[:, :, :Ncap], mx[:, :, :Ncap]


def decode(q: np.ndarray, k: np.ndarray, v: np.ndarray, seq_lens: Sequence[int], tau: np.ndarray,
           *, block_size: int, beta: float = 4.0, z: float = 1.0, a: float = 0.0,
           rescue_window: int = 128, lwb: int = 0, self_ungated: bool = False,
           screen_all: bool = False, gate_off: bool = False, bounds_only: bool = False,
           rows: Optional[Sequence[int]] = None, sel_in: Optional[np.ndarray] = None,
           summaries=None, n_threads: int = 0, quality: bool = False) -> DecodeResult:
    """One ETA decode step for every (sequence, query head), or for ``rows``.

    q [B][Hq][d]; k, v [B][Hkv][T_cap][d]; seq_lens [B]; tau [B][Hq].
    Bounds -> threshold / pins / rescue -> gated attention over the selected
    blocks plus the tail (Alg. "Hardware-Aligned Block-Sparse Decoding").
    Rows not requested are left zero.  ``bounds_only`` stops after the bounds.
    ``summaries`` = (mu, sigma, M) from ``block_index`` skips recomputing them.
    ``quality`` also gives the screening-quality diagnostics of every requested row
    (``screen_quality``) in ``blockmax``, ``quality`` and ``missed``.
    """
    q = _c(q); k = _c(k); v = _c(v)
    B, Hq, d = q.shape
    B2, Hkv, T_cap, d2 = k.shape
    assert B2 == B and d2 == d and v.shape == k.shape and v.dtype == k.dtype
    assert Hq % Hkv == 0
    b = int(block_size)
    Ncap = T_cap // b
    sl = np.ascontiguousarray(np.asarray(seq_lens, np.int32))
    tau = np.zeros((B, Hq)) if tau is None else _c(tau, np.float64).reshape(B, Hq)
    tau = np.ascontiguousarray(tau)
    rows_a = None if rows is None else np.ascontiguousarray(np.asarray(rows, np.int32))
    sel_in_a = None if sel_in is None else np.ascontiguousarray(np.asarray(sel_in, np.uint8))
    res = DecodeResult(
        o=np.zeros((B, Hq, d)),
        sel=np.zeros((B, Hq, max(Ncap, 1)), np.uint8),
        bounds=np.full((B, Hq, max(Ncap, 1)), np.nan),
        counts=np.zeros((B, Hq), np.int64),
        lse=np.full((B, Hq), -np.inf),
        rescued=np.full((B, Hq), -1, np.int64),
    )
    if quality:
        res.blockmax = np.full((B, Hq, max(Ncap, 1)), np.nan)
        res.quality = np.zeros((B, Hq, 6), np.int64)
        res.missed = np.zeros((B, Hq))
    smu = ssg = smx = None
    if summaries is not None:
        smu = np.ascontiguousarray(summaries[0], np.float64)
        ssg = np.ascontiguousarray(summaries[1], np.float64)
        smx = np.ascontiguousarray(summaries[2], np.float64)
        assert smu.shape == (B, Hkv, Ncap, d) and smx.shape == (B, Hkv, Ncap)
    P = _Problem(
        B=B, Hq=Hq, Hkv=Hkv, d=d, b=b, T_cap=T_cap,
        q_dtype=_dtype_code(q), kv_dtype=_dtype_code(k),
        q=_ptr(q), k=_ptr(k), v=_ptr(v), seq_lens=_ptr(sl), tau=_ptr(tau),
        beta=float(beta), z=float(z), a=float(a),
        c=int(rescue_window), lwb=int(lwb), self_ungated=int(bool(self_ungated)),
        screen_all=int(bool(screen_all)), gate_off=int(bool(gate_off)),
        bounds_only=int(bool(bounds_only)),
        mu=_ptr(smu), sigma=_ptr(ssg), maxnorm=_ptr(smx),
        sel_in=_ptr(sel_in_a),
        rows=_ptr(rows_a), n_rows=0 if rows_a is None else int(rows_a.shape[0]),
        n_threads=int(n_threads),
        o=_ptr(res.o), sel=_ptr(res.sel), bounds=_ptr(res.bounds), counts=_ptr(res.counts),
        lse=_ptr(res.lse), rescued=_ptr(res.rescued),
        blockmax=_ptr(res.blockmax), quality=_ptr(res.quality), missed=_ptr(res.missed),
    )
    rc = _load().eta_oracle_decode(ctypes.byref(P))
    if rc != 0:
        raise ValueError(f"eta_oracle_decode rejected the problem (code {rc})")
    res.sel = res.sel[:, :, :Ncap]
    res.bounds = res.bounds[:, :, :Ncap]
    if quality:
        res.blockmax = res.blockmax[:, :, :Ncap]
    return res


def gate_vec(S: np.ndarray, tau: float, beta: float) -> np.ndarray:
    """Elementwise ``gate`` over an array (convenience for tests)."""
    lib = _load()
    return np.array([lib.eta_oracle_gate(float(s), float(tau), float(beta)) for s in np.ravel(S)]
                    ).reshape(np.shape(S))


@dataclass
class CalibResult:
    hist: np.ndarray      # [Hq][nb] 1/t-weighted counts (not normalised)
    dens: np.ndarray      # [Hq] sum of gate * weight
    total: np.ndarray     # [Hq] sum of weights (= sequences x T)
    hist_lo: Optional[np.ndarray] = None
    hist_hi: Optional[np.ndarray] = None

    @property
    def target(self) -> np.ndarray:
        """Target density of the dynamic thresholds per head."""
        return self.dens / self.total


def calib_hist(q: np.ndarray, k: np.ndarray, tau: np.ndarray, *, beta: float, lo: float, hi: float,
               nb: int, gamma: float = 0.0, eps_abs: float = 0.0, brackets: bool = False) -> CalibResult:
    """Accumulation of Alg. "Density-Matched Offline Threshold Calibration" for every head:
    q [N][Hq][T][d], k [N][Hkv][T][d] (fp32, or bf16 as raw uint16), tau [N][Hq][T]."""
    q, k = _c(q), _c(k)
    N, Hq, T, d = q.shape
    Hkv = k.shape[1]
    assert k.shape == (N, Hkv, T, d) and Hq % Hkv == 0 and _dtype_code(q) == _dtype_code(k)
    tau = np.ascontiguousarray(np.asarray(tau, np.float64))
    assert tau.shape == (N, Hq, T)
    r = CalibResult(hist=np.zeros((Hq, nb)), dens=np.zeros(Hq), total=np.zeros(Hq))
    if brackets:
        r.hist_lo, r.hist_hi = np.zeros((Hq, nb)), np.zeros((Hq, nb))
    _load().eta_oracle_calib_hist(_ptr(q), _ptr(k), _dtype_code(q), _ptr(tau), N, Hq, Hkv, T, d,
                                  float(beta), float(lo), float(hi), int(nb), float(gamma),
                                  float(eps_abs), _ptr(r.hist), _ptr(r.hist_lo), _ptr(r.hist_hi),
                                  _ptr(r.dens), _ptr(r.total))
    return r


def calib_g(hist: np.ndarray, lo: float, hi: float, beta: float, c: float) -> float:
    """g(c) = sum_b H_b sigmoid(beta (s_b - c)) over one head's normalised histogram."""
    h = np.ascontiguousarray(np.asarray(hist, np.float64))
    return _load().eta_oracle_calib_g(_ptr(h), h.size, float(lo), float(hi), float(beta), float(c))


def calib_solve(hist: np.ndarray, lo: float, hi: float, beta: float, target: float) -> float:
    """Static threshold c of one head: g(c) = target by bisection."""
    h = np.ascontiguousarray(np.asarray(hist, np.float64))
    return _load().eta_oracle_calib_solve(_ptr(h), h.size, float(lo), float(hi), float(beta),
                                          float(target))


@dataclass
class PrefillResult:
    o: np.ndarray     # [B][Hq][T][d]
    r: np.ndarray     # [B][Hq][T]  sum of the gates over the causal keys
    lse: np.ndarray   # [B][Hq][T]  log-sum-exp of the gated scores


def prefill(q: np.ndarray, k: np.ndarray, v: np.ndarray, tau: np.ndarray, seq_lens: Sequence[int],
            *, beta: float, additive: bool = False, C: float = 0.0) -> PrefillResult:
    """Gated prefill / training forward of App. "Hardware-Aligned Forward Kernel":
    q [B][Hq][T][d], k, v [B][Hkv][T][d] (fp32, or bf16 as raw uint16), tau [B][Hq][T]."""
    q, k, v = _c(q), _c(k), _c(v)
    B, Hq, T, d = q.shape
    Hkv = k.shape[1]
    assert k.shape == (B, Hkv, T, d) and v.shape == k.shape and Hq % Hkv == 0
    assert _dtype_code(q) == _dtype_code(k) == _dtype_code(v)
    tau = np.ascontiguousarray(np.asarray(tau, np.float64))
    assert tau.shape == (B, Hq, T)
    sl = np.ascontiguousarray(np.asarray(seq_lens, np.int32))
    r = PrefillResult(o=np.zeros((B, Hq, T, d)), r=np.zeros((B, Hq, T)), lse=np.zeros((B, Hq, T)))
    _load().eta_oracle_prefill(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), _ptr(tau), _ptr(sl), B, Hq,
                               Hkv, T, d, float(beta), int(bool(additive)), float(C), _ptr(r.o),
                               _ptr(r.r), _ptr(r.lse))
    return r


def prefill_rows(q: np.ndarray, k: np.ndarray, v: np.ndarray, tau: np.ndarray,
                 seq_lens: Sequence[int], rows: np.ndarray, *, beta: float, additive: bool = False,
                 C: float = 0.0) -> PrefillResult:
    """The rows (b, h, i) of `rows` ([n][3]) of prefill(...), computed alone (same per-row
    arithmetic): o [n][d], r, lse [n].  For sampling long sequences."""
    q, k, v = _c(q), _c(k), _c(v)
    B, Hq, T, d = q.shape
    Hkv = k.shape[1]
    assert k.shape == (B, Hkv, T, d) and v.shape == k.shape and Hq % Hkv == 0
    assert _dtype_code(q) == _dtype_code(k) == _dtype_code(v)
    tau = np.ascontiguousarray(np.asarray(tau, np.float64))
    assert tau.shape == (B, Hq, T)
    rows = np.ascontiguousarray(np.asarray(rows, np.int32).reshape(-1, 3))
    assert np.all((rows[:, 0] >= 0) & (rows[:, 0] < B) & (rows[:, 1] >= 0) & (rows[:, 1] < Hq)
                  & (rows[:, 2] >= 0) & (rows[:, 2] < T))
    sl = np.ascontiguousarray(np.asarray(seq_lens, np.int32))
    n = rows.shape[0]
    r = PrefillResult(o=np.zeros((n, d)), r=np.zeros(n), lse=np.zeros(n))
    _load().eta_oracle_prefill_rows(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), _ptr(tau), _ptr(sl),
                                    B, Hq, Hkv, T, d, float(beta), int(bool(additive)), float(C),
                                    _ptr(rows), n, _ptr(r.o), _ptr(r.r), _ptr(r.lse))
    return r
