"""Comparison rules between the HIP path and the oracle (test helpers).

Masks: rows must agree on every block whose oracle score is more than EPS away
from the row's oracle boundary scores (the lowest kept and the highest dropped
non-forced score).  Top-k counts must be exactly k; forced blocks must be
present; in mass mode the count may differ by one only when the oracle's kept
mass at count-1 or count is within EPS of tau, and then only the boundary block
may differ.

Attention: max |dO| <= 2e-2 and mean |dO| <= 2e-3 over valid elements (bf16
inputs, fp32 accumulation); LSE within LSE_TOL.  The row sum adds the
probabilities after rounding to bf16 (8 significant bits, so each has a
relative error of at most 2^-8); when every probability rounds the same way
(identical keys) the sum is off by up to 2^-8 relative, i.e. ln(sum) by up to
ln(1 + 2^-8) = 3.9e-3.
"""
from __future__ import annotations

import numpy as np

EPS = 1e-5
MAX_ABS = 2e-2
MEAN_ABS = 2e-3
LSE_TOL = 4e-3


def gpu_rows(kv_idx: np.ndarray, kv_count: np.ndarray):
    """Flatten GPU outputs into a list of kept lists (row-major over B, H, nB)."""
    idx = kv_idx.reshape(-1, kv_idx.shape[-1])
    cnt = kv_count.reshape(-1)
    return [idx[r, : cnt[r]].tolist() for r in range(idx.shape[0])]


def check_idx_layout(kv_idx: np.ndarray, kv_count: np.ndarray, n_blocks: int):
    """Ascending, in range, -1 padded: exact structural checks on every row."""
    idx = kv_idx.reshape(-1, kv_idx.shape[-1])
    cnt = kv_count.reshape(-1)
    for r in range(idx.shape[0]):
        c = int(cnt[r])
        row = idx[r]
        assert 0 <= c <= row.size, (r, c)
        kept = row[:c]
        assert np.all(kept >= 0) and np.all(kept < n_blocks), (r, kept)
        assert np.all(np.diff(kept) > 0), (r, kept)
        assert np.all(row[c:] == -1), (r, row[c:])


def _softmax(s):
    w = np.exp(s - s.max())
    return w / w.sum()


def compare_masks(oracle_rows, gpu_rows_, scores: np.ndarray, mode: str, k: int = 0,
                  tau: float = 0.0, forced=(), eps: float = EPS):
    """Return (n_rows, n_identical, problems) where problems lists failing rows."""
    flat_scores = scores.reshape(-1, scores.shape[-1])
    forced = set(int(j) for j in forced)
    problems = []
    identical = 0
    for r, (ko, kg) in enumerate(zip(oracle_rows, gpu_rows_)):
        so, sg = set(ko), set(kg)
        if so == sg:
            identical += 1
            continue
        s = flat_scores[r]
        if mode == "topk" and len(kg) != k:
            problems.append((r, "count", len(kg), k))
            continue
        if not forced <= sg:
            problems.append((r, "forced missing"))
            continue
        free_kept = [j for j in ko if j not in forced]
        dropped = [j for j in range(s.size) if j not in so]
        lo = min(s[j] for j in free_kept) if free_kept else np.inf
        hi = max(s[j] for j in dropped) if dropped else -np.inf
        diff = so ^ sg
        if mode == "mass" and len(kg) != len(ko):
            if abs(len(kg) - len(ko)) != 1:
                problems.append((r, "mass count", len(kg), len(ko)))
                continue
            p = _softmax(s)
            order = sorted(free_kept, key=lambda j: (-s[j], j))
            m_forced = sum(p[j] for j in forced)
            m_all = m_forced + sum(p[j] for j in order)
            m_less = m_all - (p[order[-1]] if order else 0.0)
            if not (abs(m_all - tau) <= eps or abs(m_less - tau) <= eps):
                problems.append((r, "mass count not near tau", len(kg), len(ko), m_less, m_all))
                continue
            if len(diff) != 1:
                problems.append((r, "mass diff > 1 block", sorted(diff)))
                continue
            continue
        bad = [j for j in diff if abs(s[j] - lo) > eps and abs(s[j] - hi) > eps]
        if bad:
            problems.append((r, "blocks differ away from the boundary", bad[:5], lo, hi))
    return len(oracle_rows), identical, problems


def attention_errors(gpu_out: np.ndarray, ref: np.ndarray, valid: np.ndarray):
    """max and mean |gpu - ref| over the elements selected by `valid` (bool, same
    leading shape as ref without D)."""
    d = np.abs(gpu_out.astype(np.float64) - ref)[valid]
    return float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0


# ---- first-order remainder of dropped blocks ----
# The output is no longer a convex combination of V rows: the first-order term
# F = sum_j exp(c qbar.kbar_j) c M_j q can be several times larger than V.  It
# is formed from three factors the GPU stores in bf16 (the weights E, the
# moments M, their products T), each rounding adding at most 2^-9 relative,
# so |F| 2^-7 bounds that part; a bf16 output adds its own rounding, at most
# half a step (2^-9 |out|), bounded here by 2^-8 |out|.  The pooled keys enter
# the logits rounded to bf16, which moves a logit c q.kbar_j by at most
# c 2^-9 sum_d |q_d kbar_jd|; a log-sum-exp moves by at most its largest
# logit's change, which is added to LSE_TOL.
REM_F_REL = 2.0 ** -7
REM_OUT_REL = 2.0 ** -8

# The form of the first-order remainder the kernels compute (oracle/remainder.py):
# the block-mean query in the first-order weight.  Against the plain expansion
# (weight="query") the kernels are held to the same bounds plus the exact gap
# between the two forms, which the oracle computes.
KERNEL_REMAINDER_FORM = "block_mean"


def remainder_errors(got, ref, first, bf16_out: bool):
    """(worst excess over the elementwise bound, mean error, mean bound):
    bound = MAX_ABS + 2^-7 |F| (+ 2^-8 |ref| for bf16 outputs); the mean of the
    errors must stay under MEAN_ABS + the mean of 2^-8 |F| (+ 2^-9 |ref|)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    f = np.abs(np.asarray(first, dtype=np.float64))
    err = np.abs(got - ref)
    bound = MAX_ABS + REM_F_REL * f + (REM_OUT_REL * np.abs(ref) if bf16_out else 0.0)
    mean_bound = MEAN_ABS + np.mean(0.5 * REM_F_REL * f) + (0.5 * REM_OUT_REL * np.mean(np.abs(ref)) if bf16_out else 0.0)
    return float(np.max(err - bound)), float(np.mean(err)), float(mean_bound)


def remainder_errors_vs_plain(got, ref_plain, ref_kernel_form, first, bf16_out: bool):
    """remainder_errors against the plain expansion, each element's bound
    widened by |ref_kernel_form - ref_plain| (the first-order weight taken at
    the block-mean query instead of the query's own)."""
    gap = np.abs(np.asarray(ref_kernel_form, dtype=np.float64) - np.asarray(ref_plain, dtype=np.float64))
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - np.asarray(ref_plain, dtype=np.float64))
    f = np.abs(np.asarray(first, dtype=np.float64))
    bound = MAX_ABS + REM_F_REL * f + gap + (REM_OUT_REL * np.abs(ref_plain) if bf16_out else 0.0)
    return float(np.max(err - bound)), float(np.mean(gap)), float(np.max(gap))


def remainder_lse_bound(q, kbar, scale):
    """Per query: LSE_TOL + c 2^-9 max_j sum_d |q_d kbar_jd|."""
    q = np.abs(np.asarray(q, dtype=np.float64))
    kb = np.abs(np.asarray(kbar, dtype=np.float64))
    return LSE_TOL + scale * 2.0 ** -9 * np.max(q @ kb.T, axis=1)
