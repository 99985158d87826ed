"""Brute-force NumPy reading of the ETA decode step, for tiny inputs only.

An independent second reading of Alg. "Hardware-Aligned Block-Sparse Decoding
(Inference)": the full blocks are cut into chunks of ``c`` blocks; each chunk
keeps its own online-softmax state (m, l, acc); the first chunk tracks the block
with the largest bound and, if it attended nothing, admits that block (top-1
rescue); the last chunk attends the partial tail; a final pass merges the chunk
states by the associative log-sum-exp rule.  Summaries come from numpy's
mean / population variance / norm, and the gate uses scipy's logistic function,
so nothing is shared with the C oracle.

Reading for T < b (the algorithm would run zero chunks): a single chunk that
only attends the tail.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import expit


def _to_f64(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def decode_head(q, K, V, T, b, c, tau, *, a=0.0, z=1.0, beta=4.0, lwb=0, self_ungated=False):
    """Returns (o, attended_block_set, attended_token_count) for one query head."""
    q = _to_f64(np.asarray(q)); K = _to_f64(np.asarray(K))[:T]; V = _to_f64(np.asarray(V))[:T]
    d = q.shape[0]
    s = 1.0 / math.sqrt(d)
    N = T // b
    tau_eff = tau - a
    qn = math.sqrt(float(q @ q))

    def bound(j):
        blk = K[j * b:(j + 1) * b]
        mu = blk.mean(axis=0)
        var = blk.var(axis=0)                   # population variance (ddof = 0)
        M = np.linalg.norm(blk, axis=1).max()
        return s * min(float(q @ mu) + z * math.sqrt(float((q * q) @ var)), qn * M)

    def gated(idx):
        S = s * (K[idx] @ q)
        g = S * expit(beta * (S - tau_eff)) if not (math.isinf(tau_eff) and tau_eff < 0) else S
        if self_ungated:
            g = np.where(idx == T - 1, S, g)
        return g

    def update(state, idx):
        m, l, acc = state
        St = gated(idx)
        m_new = max(m, float(St.max()))
        alpha = math.exp(m - m_new) if m != -math.inf else 0.0
        p = np.exp(St - m_new)
        return (m_new, l * alpha + float(p.sum()), acc * alpha + p @ V[idx])

    n_chunks = max(1, -(-N // c)) if c > 0 else 1
    if c <= 0:
        c_eff = max(N, 1)
    else:
        c_eff = c
    mids = []
    attended = set()
    tokens = 0
    for kc in range(n_chunks):
        st = (-math.inf, 0.0, np.zeros(d))
        n_att = 0
        best, best_j = -math.inf, -1
        for j in range(kc * c_eff, min((kc + 1) * c_eff, N)):
            bj = bound(j)
            if bj >= tau_eff or j >= N - lwb:
                st = update(st, np.arange(j * b, (j + 1) * b))
                attended.add(j)
                n_att += b
                tokens += b
            if kc == 0 and c > 0 and bj > best:
                best, best_j = bj, j
        if kc == 0 and c > 0 and n_att == 0 and best_j >= 0:
            st = update(st, np.arange(best_j * b, (best_j + 1) * b))
            attended.add(best_j)
            tokens += b
        if kc == n_chunks - 1 and T > N * b:
            st = update(st, np.arange(N * b, T))
            tokens += T - N * b
        mids.append(st)
    # global reduction across chunks
    mg, lg, og = -math.inf, 0.0, np.zeros(d)
    for m, l, acc in mids:
        if m == -math.inf:
            continue
        mn = max(mg, m)
        ag = math.exp(mg - mn) if mg != -math.inf else 0.0
        ac = math.exp(m - mn)
        lg = lg * ag + l * ac
        og = og * ag + acc * ac
        mg = mn
    o = og / lg if lg > 0 else np.zeros(d)
    return o, attended, tokens
