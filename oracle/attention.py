"""Block-sparse and dense softmax attention (oracle; test infrastructure only).

Section 4.2.2 of the paper: the kept ("critical") blocks are computed exactly.
Reading taken here: for a query token n in query block i, attention runs over the
valid key tokens of the kept KV blocks of row i only; the softmax is normalised
over those keys (non-kept blocks contribute nothing -- the paper's Taylor
remainder for them is not defined in its text).  The dense fallback of
Appendix A.2.2 is the same with every block kept.

This is the plain two-pass definition, not an online softmax:
    l[m]   = c * <Q[n], K[m]>              over kept keys m
    M      = max_m l[m]
    w[m]   = exp(l[m] - M)
    O[n]   = sum_m w[m] V[m] / sum_m w[m]
    LSE[n] = M + ln(sum_m w[m])            (natural log)
"""
from __future__ import annotations

import numpy as np

from .blocks import block_bounds


def _attend(qrows: np.ndarray, keys: np.ndarray, vals: np.ndarray, scale: float):
    logits = scale * (qrows @ keys.T)
    mx = logits.max(axis=1, keepdims=True)
    w = np.exp(logits - mx)
    denom = w.sum(axis=1, keepdims=True)
    out = (w @ vals) / denom
    lse = mx[:, 0] + np.log(denom[:, 0])
    return out, lse


def block_sparse_attention(q, k, v, kept, block: int, scale: float, rows=None):
    """Attention of every (b, h, query block) over its kept KV blocks.

    q, k, v : float64 [B, H, N, D]
    kept    : kept[b][h][i] = iterable of KV block indices (any order)
    rows    : optional iterable of (b, h, i); only those query blocks are
              computed, the rest of the output stays NaN
    returns (out float64 [B, H, N, D], lse float64 [B, H, N])
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, H, N, D = q.shape
    bounds = block_bounds(N, block)
    out = np.full((B, H, N, D), np.nan)
    lse = np.full((B, H, N), np.nan)
    if rows is None:
        rows = [(b, h, i) for b in range(B) for h in range(H) for i in range(len(bounds))]
    for b, h, i in rows:
        qa, qb = bounds[i]
        blocks = [int(j) for j in kept[b][h][i]]
        if not blocks:
            out[b, h, qa:qb] = 0.0
            lse[b, h, qa:qb] = -np.inf
            continue
        key_tok = np.concatenate([np.arange(*bounds[j]) for j in blocks])
        o, s = _attend(q[b, h, qa:qb], k[b, h, key_tok], v[b, h, key_tok], scale)
        out[b, h, qa:qb] = o
        lse[b, h, qa:qb] = s
    return out, lse


def dense_attention(q, k, v, scale: float, rows=None, block: int = 64):
    """Full softmax attention over all N keys (the dense fallback).

    rows: optional iterable of (b, h, i) query blocks of size `block` to compute.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, H, N, D = q.shape
    out = np.full((B, H, N, D), np.nan)
    lse = np.full((B, H, N), np.nan)
    bounds = block_bounds(N, block)
    if rows is None:
        rows = [(b, h, i) for b in range(B) for h in range(H) for i in range(len(bounds))]
    for b, h, i in rows:
        qa, qb = bounds[i]
        o, s = _attend(q[b, h, qa:qb], k[b, h], v[b, h], scale)
        out[b, h, qa:qb] = o
        lse[b, h, qa:qb] = s
    return out, lse
