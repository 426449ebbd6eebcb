"""Block-importance scoring and block-mask construction (oracle; test
infrastructure only).

Section 4.2.2 of the paper routes attention by a block-wise similarity score and
keeps the "critical" blocks; Appendix A.2.2 runs it at density 0.1 with block 64
("score-based routing").  The paper does not print the score or the rule; this
oracle implements the reading:

  score      s[i, j] = c * <qbar_i, kbar_j>,   c = softmax scale (1/sqrt(D) default)
  top-k      keep the k blocks j with the largest s[i, j]; ties go to the lower j;
             k = clamp(ceil(r * nB - 1e-6), 1, nB) from a keep ratio r, or given.
  mass       p[i, :] = softmax over all j of s[i, :]; the forced set F (blocks that
             hold any token of frame t = 0) is kept first and its mass counts;
             then blocks outside F are added in (s desc, j asc) order while the
             kept mass is below tau and fewer than `cap` blocks are kept,
             cap = clamp(ceil(rho * nB - 1e-6), |F|, nB).
  output     kept blocks in ascending order.
"""
from __future__ import annotations

import math

import numpy as np

_EPS_COUNT = 1e-6


def block_scores(q_pool: np.ndarray, k_pool: np.ndarray, scale: float) -> np.ndarray:
    """s[..., i, j] = scale * sum_d q_pool[..., i, d] * k_pool[..., j, d]  (float64)."""
    q = np.asarray(q_pool, dtype=np.float64)
    k = np.asarray(k_pool, dtype=np.float64)
    return scale * np.matmul(q, np.swapaxes(k, -1, -2))


def topk_count(n_blocks: int, keep_ratio: float = 0.0, topk: int = 0) -> int:
    """Blocks kept per query block in top-k mode."""
    if topk and topk > 0:
        k = int(topk)
    else:
        k = math.ceil(float(keep_ratio) * n_blocks - _EPS_COUNT)
    return max(1, min(n_blocks, k))


def _order_desc(row: np.ndarray, candidates) -> list:
    """Candidates sorted by (score descending, block index ascending)."""
    cand = np.asarray(list(candidates), dtype=np.int64)
    if cand.size == 0:
        return []
    # lexsort sorts by the last key first: primary -score, secondary index.
    order = np.lexsort((cand, -row[cand]))
    return [int(j) for j in cand[order]]


def select_topk(scores: np.ndarray, k: int):
    """Per row: the k best blocks, as an ascending list.

    scores: [..., nB, nB]; returns a nested list with the leading shape, each
    leaf an ascending list of kept block indices.
    """
    scores = np.asarray(scores, dtype=np.float64)
    lead = scores.shape[:-1]
    nb = scores.shape[-1]
    flat = scores.reshape(-1, nb)
    rows = []
    for r in range(flat.shape[0]):
        best = _order_desc(flat[r], range(nb))[:k]
        rows.append(sorted(best))
    return _reshape_nested(rows, lead)


def first_frame_blocks(grid_h: int, grid_w: int, block: int, n_blocks: int) -> list:
    """Blocks holding at least one token of frame t = 0 (tokens 0 .. H*W-1)."""
    frame = int(grid_h) * int(grid_w)
    return [j for j in range(n_blocks) if j * block < frame]


def mass_cap(n_blocks: int, max_keep_ratio: float, n_forced: int) -> int:
    """Upper bound on kept blocks per row in mass mode (never below |F|)."""
    cap = math.ceil(float(max_keep_ratio) * n_blocks - _EPS_COUNT)
    return max(n_forced, min(n_blocks, cap))


def select_cummass(scores: np.ndarray, tau: float, cap: int, forced=()):
    """Per row: forced blocks plus the best other blocks until the kept softmax
    mass reaches tau or `cap` blocks are kept.  Returns ascending lists."""
    scores = np.asarray(scores, dtype=np.float64)
    lead = scores.shape[:-1]
    nb = scores.shape[-1]
    flat = scores.reshape(-1, nb)
    forced = sorted(set(int(j) for j in forced))
    forced_set = set(forced)
    others = [j for j in range(nb) if j not in forced_set]
    rows = []
    for r in range(flat.shape[0]):
        s = flat[r]
        w = np.exp(s - s.max())
        p = w / w.sum()
        kept = list(forced)
        mass = float(p[forced].sum()) if forced else 0.0
        for j in _order_desc(s, others):
            if mass >= tau or len(kept) >= cap:
                break
            kept.append(j)
            mass += float(p[j])
        rows.append(sorted(kept))
    return _reshape_nested(rows, lead)


def kept_to_arrays(kept, n_blocks: int, kmax: int):
    """Nested kept lists -> (kv_idx int32 [..., nB, kmax] padded with -1,
    kv_count int32 [..., nB])."""
    flat, lead = _flatten_nested(kept)
    idx = np.full((len(flat), kmax), -1, dtype=np.int32)
    cnt = np.zeros(len(flat), dtype=np.int32)
    for r, row in enumerate(flat):
        if len(row) > kmax:
            raise ValueError(f"row {r} keeps {len(row)} blocks > kmax {kmax}")
        idx[r, : len(row)] = row
        cnt[r] = len(row)
    return idx.reshape(lead + (kmax,)), cnt.reshape(lead)


def kept_to_mask(kept, n_blocks: int) -> np.ndarray:
    """Nested kept lists -> uint8 mask [..., nB, nB] (1 = kept)."""
    flat, lead = _flatten_nested(kept)
    m = np.zeros((len(flat), n_blocks), dtype=np.uint8)
    for r, row in enumerate(flat):
        m[r, row] = 1
    return m.reshape(lead + (n_blocks,))


def _reshape_nested(rows: list, lead: tuple):
    if len(lead) == 1:
        return rows
    step = int(np.prod(lead[1:]))
    return [_reshape_nested(rows[i * step:(i + 1) * step], lead[1:]) for i in range(lead[0])]


def _flatten_nested(kept):
    """Flatten nested lists whose leaves are lists of ints; return (rows, lead)."""
    lead = []
    node = kept
    while isinstance(node, list) and node and isinstance(node[0], list):
        lead.append(len(node))
        node = node[0]
    lead = tuple(lead)
    rows = []

    def walk(n, depth):
        if depth == len(lead):
            rows.append(list(n))
        else:
            for c in n:
                walk(c, depth + 1)

    walk(kept, 0)
    return rows, lead
