"""Pure-Python brute force for tiny inputs (test infrastructure only).

It works on the *logical* per-sequence K/V (position p of sequence b, before
any paging or ring placement), builds the visible position set explicitly,
materialises a -inf mask over every position of the sequence and evaluates
softmax attention with Python floats.  Storage values are decoded with
torch's own dtype conversions, so this path shares neither the C oracle's
decoders nor its address arithmetic.

Verify (Sec. 2: the k+1 tokens of a round are scored in one parallel target
pass): query i of sequence b sees positions {0, ..., n_b - k + i - 1}.
Draft (Sec. 3.1 / Sec. 4: StreamingLLM sinks plus sliding window): with m_b
positions, visible = {p < S} U {p >= m_b - W}, intersected with {p < m_b}.
"""
from __future__ import annotations

import math
from typing import Optional

import numpy as np
import torch


def _f64(t: torch.Tensor, scale: Optional[torch.Tensor] = None, head_axis: int = 1) -> np.ndarray:
    x = t.detach().cpu().to(torch.float64)
    if scale is not None:
        shape = [1] * x.dim()
        shape[head_axis] = -1
        x = x * scale.detach().cpu().to(torch.float64).view(shape)
    return x.numpy()


def _attend(qrow, keys, vals, allowed):
    """Masked softmax attention of one query over all positions of a sequence."""
    n = len(keys)
    scores = []
    for p in range(n):
        if p in allowed:
            scores.append(sum(a * b for a, b in zip(qrow, keys[p])))
        else:
            scores.append(-math.inf)
    # a NaN score makes the maximum NaN (Python's max() would depend on where
    # the NaN sits), and with it every weight: the row is NaN
    if any(s != s for s in scores):
        M = math.nan
    else:
        M = max(scores) if scores else -math.inf
    if M == -math.inf:  # no visible key, or every visible score is -inf (weighs zero)
        return [0.0] * len(qrow), -math.inf
    w = [math.exp(s - M) for s in scores]
    L = sum(w)
    out = [sum(w[p] * vals[p][d] for p in range(n)) / L for d in range(len(vals[0]))]
    return out, M + math.log(L)


def verify(q, logical_k, logical_v, kv_lens, k, sm_scale, k_scale=None, v_scale=None):
    """q [B, k+1, Hq, D]; logical K/V [B, Hkv, nmax, D] (storage dtype)."""
    Q = _f64(q)
    K = _f64(logical_k, k_scale)
    V = _f64(logical_v, v_scale)
    B, nq, Hq, D = Q.shape
    Hkv = K.shape[1]
    g = Hq // Hkv
    out = np.zeros((B, nq, Hq, D))
    lse = np.zeros((B, nq, Hq))
    for b in range(B):
        n = int(kv_lens[b])
        for i in range(nq):
            allowed = set(range(0, n - k + i))
            for h in range(Hq):
                hk = h // g
                keys = [[sm_scale * x for x in K[b, hk, p]] for p in range(n)]
                vals = [list(V[b, hk, p]) for p in range(n)]
                o, l = _attend(list(Q[b, i, h]), keys, vals, allowed)
                out[b, i, h] = o
                lse[b, i, h] = l
    return out, lse


def draft(q, logical_k, logical_v, seq_lens, S, W, sm_scale, k_scale=None, v_scale=None):
    """q [B, Hq, D]; logical K/V [B, Hkv, >= m_b, D]: attention over sinks + window."""
    Q = _f64(q)
    K = _f64(logical_k, k_scale)
    V = _f64(logical_v, v_scale)
    B, Hq, D = Q.shape
    Hkv = K.shape[1]
    g = Hq // Hkv
    out = np.zeros((B, Hq, D))
    lse = np.zeros((B, Hq))
    for b in range(B):
        m = int(seq_lens[b])
        allowed = set(p for p in range(m) if p < S or p >= m - W)
        for h in range(Hq):
            hk = h // g
            keys = [[sm_scale * x for x in K[b, hk, p]] for p in range(m)]
            vals = [list(V[b, hk, p]) for p in range(m)]
            o, l = _attend(list(Q[b, h]), keys, vals, allowed)
            out[b, h] = o
            lse[b, h] = l
    return out, lse
