"""Seeded synthetic decode workloads for the ETA decode path.

This module is shared by the tests, the smoke check and the benchmark.  It holds
random draws and data layout only -- none of the method's arithmetic.  The
paper's speed workloads (real long-context text on a trained model) are not
available, so query-aligned "planted" blocks stand in for the salient context:
a planted block's keys are ``3 sqrt(d) u + N(0, 1)`` with ``u`` the unit
direction of the query (MHA) or of the sum of the group's queries (GQA), so all
heads of the group see it.  Everything else is ``N(0, 1)``.

Data layout (what the GPU library and the oracle both consume):
  q        [B][Hq][d]             float32 or bfloat16
  k, v     [B][Hkv][T_cap][d]     float32 or bfloat16, token rows contiguous
  seq_lens [B]                    int32
  W        [Hq*d][Hq] float32     predictor weights (None in constant mode)
  bias     [Hq] float32           predictor bias, or the frozen constants
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np
import torch

# Rescue window per block size: the paper's best chunk arms (b=64 -> c=128,
# b=128 -> c=64), App. "Chunked Decoding and Two-Stage Reduction".
RESCUE_WINDOW = {64: 128, 128: 64}


@dataclass
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    d: int
    block: int
    T_cap: int
    seq_lens: List[int]
    dtype: torch.dtype
    q: torch.Tensor
    k: torch.Tensor
    v: torch.Tensor
    W: Optional[torch.Tensor]          # None: constant (frozen) thresholds
    bias: torch.Tensor                 # predictor bias or frozen per-head constants
    beta: float = 4.0
    z: float = 1.0
    a: float = 0.0
    rescue_window: int = 128
    lwb: int = 0
    target_survival: Optional[float] = None
    planted: dict = field(default_factory=dict)   # (b, kv head) -> sorted planted block ids

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def n_blk_cap(self) -> int:
        return self.T_cap // self.block

    @property
    def W_heads(self) -> Optional[torch.Tensor]:
        """W in the library's head-major layout [Hq][Hq d] (row h: the weights of
        head h's threshold), i.e. W transposed."""
        return None if self.W is None else self.W.t().contiguous()

    def to(self, device) -> "Workload":
        out = Workload(**{f: getattr(self, f) for f in self.__dataclass_fields__})
        for n in ("q", "k", "v", "W", "bias"):
            t = getattr(self, n)
            setattr(out, n, None if t is None else t.to(device))
        return out


def _planted_positions(rng: np.random.Generator, N: int, spec: dict) -> np.ndarray:
    """Block ids to plant for one (sequence, head): 'frac' uniform, or 'start'/'end'/'random' fractions."""
    if N <= 0:
        return np.zeros(0, np.int64)
    ids = set()
    if "count" in spec:
        n = min(int(spec["count"]), N)
        ids.update(rng.choice(N, size=n, replace=False).tolist())
    if "frac" in spec:
        n = min(int(round(spec["frac"] * N)), N)
        ids.update(rng.choice(N, size=n, replace=False).tolist())
    if "start" in spec:
        n = min(int(math.ceil(spec["start"] * N)), N)
        ids.update(range(n))
    if "end" in spec:
        n = min(int(math.ceil(spec["end"] * N)), N)
        ids.update(range(N - n, N))
    if "random" in spec:
        rest = np.array(sorted(set(range(N)) - ids), np.int64)
        n = min(int(math.ceil(spec["random"] * N)), rest.shape[0])
        if n > 0:
            ids.update(rng.choice(rest, size=n, replace=False).tolist())
    return np.array(sorted(ids), np.int64)


def make_workload(*, name: str = "custom", B: int, Hq: int, Hkv: int, d: int, block: int,
                  seq_lens: Sequence[int], T_cap: Optional[int] = None,
                  dtype: torch.dtype = torch.bfloat16, planted: Optional[dict] = None,
                  per_head_planting: bool = False, predictor: bool = True,
                  w_std: float = 0.02, tau_const=None, beta: float = 4.0, z: float = 1.0,
                  a: float = 0.0, rescue_window: Optional[int] = None, lwb: int = 0,
                  target_survival: Optional[float] = None, seed: int = 0,
                  device="cpu") -> Workload:
    """Draw one seeded workload.

    Noise tensors come from a torch generator on ``device`` (so the same seed on a
    different device type gives different, equally valid data); block positions
    and constants come from a numpy generator and do not depend on the device.
    """
    seq_lens = [int(t) for t in seq_lens]
    if T_cap is None:
        T_cap = max(seq_lens) if seq_lens else 0
    assert len(seq_lens) == B and Hq % Hkv == 0
    G = Hq // Hkv
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    rng = np.random.default_rng(seed)

    q32 = torch.randn(B, Hq, d, generator=gen, device=dev, dtype=torch.float32)
    q = q32.to(dtype)
    k = torch.empty(B, Hkv, T_cap, d, device=dev, dtype=dtype)
    v = torch.empty(B, Hkv, T_cap, d, device=dev, dtype=dtype)
    qs = q.float()
    planted_ids = {}
    for bb in range(B):
        N = seq_lens[bb] // block
        for g in range(Hkv):
            kk = torch.randn(T_cap, d, generator=gen, device=dev, dtype=torch.float32)
            if planted:
                ids = _planted_positions(rng, N, planted)
                planted_ids[(bb, g)] = ids
                if per_head_planting:
                    # MHA-style: each head of the group gets its own direction (G == 1 in config 1)
                    u = qs[bb, g * G] / qs[bb, g * G].norm()
                else:
                    s = qs[bb, g * G:(g + 1) * G].sum(0)
                    u = s / s.norm()
                if ids.size:
                    rows = (torch.as_tensor(ids, device=dev)[:, None] * block
                            + torch.arange(block, device=dev)[None, :]).reshape(-1)
                    kk[rows] += 3.0 * math.sqrt(d) * u
            k[bb, g] = kk.to(dtype)
            v[bb, g] = torch.randn(T_cap, d, generator=gen, device=dev, dtype=torch.float32).to(dtype)
            del kk

    if predictor:
        W = (torch.randn(Hq * d, Hq, generator=gen, device=dev, dtype=torch.float32) * w_std)
        bias = torch.zeros(Hq, device=dev, dtype=torch.float32)
    else:
        W = None
        if tau_const is None:
            raise ValueError("constant-threshold mode needs tau_const")
        if isinstance(tau_const, tuple):      # (lo, hi): per-head uniform draw
            lo, hi = tau_const
            vals = rng.uniform(lo, hi, size=Hq)
        else:
            vals = np.full(Hq, float(tau_const))
        bias = torch.as_tensor(vals, dtype=torch.float32, device=dev)
    if rescue_window is None:
        rescue_window = RESCUE_WINDOW.get(block, 128)
    return Workload(name=name, B=B, Hq=Hq, Hkv=Hkv, d=d, block=block, T_cap=T_cap,
                    seq_lens=seq_lens, dtype=dtype, q=q, k=k, v=v, W=W, bias=bias, beta=beta,
                    z=z, a=a, rescue_window=rescue_window, lwb=lwb,
                    target_survival=target_survival, planted=planted_ids)


# ------------------------------------------------------------ the five configs

def config1(device="cpu", seed: int = 1) -> Workload:
    """B=1, 4 heads MHA, d=64, T=4096, b=64, fp32; 8 planted blocks per head; tau=2.0, beta=4."""
    return make_workload(name="c1_mha_4k_fp32", B=1, Hq=4, Hkv=4, d=64, block=64,
                         seq_lens=[4096], dtype=torch.float32, planted={"count": 8},
                         per_head_planting=True, predictor=False, tau_const=2.0, beta=4.0,
                         z=1.0, seed=seed, device=device)


def config2(device="cpu", seed: int = 2) -> Workload:
    """B=1, 16/4 GQA, d=128, T=32768, b=64, bf16; 5% planted; predictor at ~10% survival."""
    return make_workload(name="c2_gqa_32k", B=1, Hq=16, Hkv=4, d=128, block=64,
                         seq_lens=[32768], planted={"frac": 0.05}, predictor=True, z=1.0,
                         target_survival=0.10, seed=seed, device=device)


def config3(device="cpu", seed: int = 3) -> Workload:
    """B=8, 16/4 GQA, d=128, T=131072, b=64, bf16; planted first/last 2% + 3% random; ~10%."""
    return make_workload(name="c3_gqa_128k_b8", B=8, Hq=16, Hkv=4, d=128, block=64,
                         seq_lens=[131072] * 8,
                         planted={"start": 0.02, "end": 0.02, "random": 0.03},
                         predictor=True, z=1.0, target_survival=0.10, seed=seed, device=device)


def config4(device="cpu", seed: int = 4, survival: float = 0.20) -> Workload:
    """B=1, 16/4 GQA, d=128, T=524288, b=128, bf16; 1% planted; survival swept by the bias."""
    return make_workload(name="c4_gqa_512k", B=1, Hq=16, Hkv=4, d=128, block=128,
                         seq_lens=[524288], planted={"frac": 0.01}, predictor=True, z=1.0,
                         target_survival=survival, seed=seed, device=device)


def config5(device="cpu", seed: int = 5, predictor: bool = False) -> Workload:
    """B=32 ragged T~U[16384, 65536], 32/8 GQA, d=128, b=64, bf16, pure N(0,1);
    constants U[1.5, 3.0] per head with z=2 (calibrated mode), or predictor at ~10%."""
    rng = np.random.default_rng(seed + 1000)
    lens = rng.integers(16384, 65536, size=32, endpoint=True).tolist()
    if predictor:
        return make_workload(name="c5_ragged_pred", B=32, Hq=32, Hkv=8, d=128, block=64,
                             seq_lens=lens, T_cap=65536, planted=None, predictor=True, z=2.0,
                             target_survival=0.10, seed=seed, device=device)
    return make_workload(name="c5_ragged_const", B=32, Hq=32, Hkv=8, d=128, block=64,
                         seq_lens=lens, T_cap=65536, planted=None, predictor=False,
                         tau_const=(1.5, 3.0), z=2.0, seed=seed, device=device)


CONFIGS = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5}


# ------------------------------------------------------------ threshold placement

def place_bias(bounds: np.ndarray, n_blocks: Sequence[int], qW: np.ndarray, target: float,
               a: float = 0.0) -> np.ndarray:
    """Predictor bias that makes about ``target`` of each head's full blocks survive.

    ``bounds`` [B][Hq][N_cap] are screening bounds computed elsewhere (by the
    oracle in tests, by the GPU path in the benchmark); ``qW`` [B][Hq] is the
    predictor output with zero bias.  Sequence b's effective threshold for head
    h is qW[b, h] + bias[h] - a, so a block survives iff bound - qW[b, h] >=
    bias[h] - a.  Per head, bias - a is put midway between the k-th and
    (k+1)-th largest of bound - qW[b, h] pooled over the batch's full blocks
    (k = ceil(target * n)): exactly k blocks of the batch survive and no bound
    sits at its threshold.  (Each sequence's predictor output shifts its own
    threshold, so the survival of single sequences still varies.)
    """
    bounds = np.asarray(bounds, np.float64)
    qW = np.asarray(qW, np.float64)
    B, Hq, _ = bounds.shape
    bias = np.zeros(Hq, np.float64)
    for h in range(Hq):
        vals = np.concatenate([bounds[b, h, :n_blocks[b]] - qW[b, h] for b in range(B)])
        vals = np.sort(vals[np.isfinite(vals)])[::-1]
        n = vals.shape[0]
        if n == 0:
            t = 0.0
        else:
            kk = int(math.ceil(target * n))
            if kk >= n:
                t = vals[-1] - 1.0
            elif kk <= 0:
                t = vals[0] + 1.0
            else:
                t = 0.5 * (vals[kk - 1] + vals[kk])
        bias[h] = t + a
    return bias.astype(np.float32)


def as_numpy(t: torch.Tensor) -> np.ndarray:
    """CPU numpy view of a tensor: float32 stays float32, bfloat16 becomes its raw uint16 bits."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.numpy()
    raise TypeError(f"unsupported dtype {t.dtype}")


@dataclass
class CalibStream:
    """Calibration split for the offline threshold calibration: N sequences of T
    steps, the query of every step, the keys, and the dynamic thresholds the
    deployed predictor produced at each step."""
    q: torch.Tensor      # bf16 [N][Hq][T][d]
    k: torch.Tensor      # bf16 [N][Hkv][T][d]
    tau: torch.Tensor    # fp32 [N][Hq][T]


def calib_stream(*, N: int, Hq: int, Hkv: int, T: int, d: int, seed: int = 0,
                 tau_mean=(0.5, 2.0), tau_std: float = 0.3, planted_frac: float = 0.05,
                 tau_const: Optional[Sequence[float]] = None, device="cpu") -> CalibStream:
    """q, k ~ N(0, 1) in fp32 rounded to bf16; a fraction of keys planted along the
    group's mean query direction (3 sqrt(d) u + N(0, 1)) so the score stream has a
    right tail; per-head dynamic thresholds N(mu_h, tau_std) per step with mu_h
    spread over tau_mean, or exactly tau_const[h] at every step."""
    # large streams are drawn on the device (its own seeded generator)
    gdev = torch.device(device) if N * Hq * T * d > (1 << 26) else torch.device("cpu")
    gen = torch.Generator(device=gdev).manual_seed(seed)
    q = torch.randn(N, Hq, T, d, generator=gen, device=gdev)
    k = torch.randn(N, Hkv, T, d, generator=gen, device=gdev)
    G = Hq // Hkv
    u = q.view(N, Hkv, G, T, d).sum(dim=(2, 3))
    u = u / u.norm(dim=-1, keepdim=True)
    plant = torch.rand(N, Hkv, T, generator=gen, device=gdev) < planted_frac
    k = torch.where(plant[..., None], 3.0 * math.sqrt(d) * u[:, :, None, :] + k, k)
    if tau_const is not None:
        tau = torch.tensor(list(tau_const), dtype=torch.float32,
                           device=gdev)[None, :, None].expand(N, Hq, T)
    else:
        mu = torch.linspace(tau_mean[0], tau_mean[1], Hq, device=gdev)
        tau = mu[None, :, None] + tau_std * torch.randn(N, Hq, T, generator=gen, device=gdev)
    return CalibStream(q=q.to(torch.bfloat16).to(device), k=k.to(torch.bfloat16).to(device),
                       tau=tau.to(torch.float32).contiguous().to(device))
