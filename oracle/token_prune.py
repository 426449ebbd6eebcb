"""feat_norm token pruning (oracle; test infrastructure only).

Section 4.2.3 describes token pruning as dropping redundant latent tokens so
that later attention and feed-forward work runs on fewer tokens, with the
criterion, the ratio and the reconstruction rule tuned per model; Appendix
A.2.2 keeps 50% of the video tokens by the "feat_norm" saliency score in the
LTX-2.3 refinement stage.  The paper gives no formula; readings taken here
(the design notes list them):

* saliency of token n of batch entry b: its hidden state's squared L2 norm
  over the channel dimension, sum_c x[b, n, c]^2 (ranking by the norm or by
  its square is the same order);
* k = clamp(ceil(r * N - 1e-6), 1, N) tokens are kept per batch entry: the k
  largest scores, ties to the lower token index, listed in ascending order;
* gather: the kept rows, in that order;
* scatter (reconstruction): the processed kept rows go back to their
  positions and every dropped token keeps its input row.
"""
from __future__ import annotations

import math

import numpy as np

_EPS_COUNT = 1e-6


def token_scores(x: np.ndarray) -> np.ndarray:
    """x [B, N, C] -> float64 [B, N]: sum over c of x^2."""
    x = np.asarray(x, dtype=np.float64)
    return np.sum(x * x, axis=-1)


def keep_count(n_tokens: int, keep_ratio: float) -> int:
    k = math.ceil(float(keep_ratio) * n_tokens - _EPS_COUNT)
    return max(1, min(int(n_tokens), k))


def select_tokens(scores: np.ndarray, k: int) -> np.ndarray:
    """scores [B, N] -> int64 [B, k]: per row the k best tokens (score
    descending, index ascending among equals), returned in ascending order."""
    scores = np.asarray(scores, dtype=np.float64)
    B, N = scores.shape
    out = np.empty((B, k), dtype=np.int64)
    idx = np.arange(N)
    for b in range(B):
        order = np.lexsort((idx, -scores[b]))       # primary: -score, then index
        out[b] = np.sort(order[:k])
    return out


def gather_tokens(x: np.ndarray, kept: np.ndarray) -> np.ndarray:
    """x [B, N, C], kept [B, k] -> [B, k, C]."""
    x = np.asarray(x)
    return np.stack([x[b, kept[b]] for b in range(x.shape[0])])


def scatter_tokens(y_kept: np.ndarray, kept: np.ndarray, base: np.ndarray) -> np.ndarray:
    """Rows of y_kept [B, k, C] back to positions kept [B, k]; every other row
    of the result is base [B, N, C]."""
    out = np.array(base, copy=True)
    for b in range(out.shape[0]):
        out[b, kept[b]] = y_kept[b]
    return out
