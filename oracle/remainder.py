"""First-order remainder for the key blocks a query block does not keep
(oracle; test infrastructure only).

Section 4.2.2 (and the summary of piecewise sparse attention in Section 2)
describes the non-critical blocks as compensated by a first-order Taylor
approximation rather than dropped; the paper states no formula.  The
definition taken here is the plain first-order expansion of each dropped key's
exponential about its block's mean key.

For query token n (query q = Q[n]) of query block i and a key block j that row
i does not keep (valid tokens t, n_j of them, means kbar_j and vbar_j,
deviations dk_t = K[t] - kbar_j):

    exp(c q.K[t]) = exp(c q.kbar_j) * exp(c q.dk_t)
                 ~ exp(c q.kbar_j) * (1 + c q.dk_t)          (first order in dk_t)

Summed over the block, with sum_t dk_t = 0:

    weight_j = n_j exp(c q.kbar_j)
    value_j  = exp(c q.kbar_j) (n_j vbar_j + c M_j q)
    M_j[e, d] = sum_t V[t, e] dk_t[d]                 (the block's moment)

and the output adds these to the exact sums over the kept keys m:

    O[n]   = (sum_m exp(c q.K[m]) V[m] + sum_j value_j)
             / (sum_m exp(c q.K[m]) + sum_j weight_j)
    LSE[n] = ln(denominator)

Its error against dense attention is second order in the key deviations alone,
whatever the queries are.

weight="block_mean" gives the cheaper second approximation the GPU kernels
compute: in the first-order term only, exp(c q.kbar_j) is replaced by
exp(c qbar_i.kbar_j) with qbar_i the block-mean query, so that the term becomes
one matrix per query block, T_i = sum_j exp(c qbar_i.kbar_j) M_j, applied to
every query of the block.  That replacement is exact when the block's queries
equal their mean and otherwise changes each first-order term by the relative
amount exp(c (qbar_i - q).kbar_j) - 1, which is of order one when the queries
of a block differ by order one: the error of this form against dense attention
is then first order in the key deviations (a product of a query and a key
deviation), not second.  The zero-order weight and value keep the query's own
logit in both forms, so the two forms share the denominator.

A block is dropped for row i when no in-range entry of the row's list names
it; the kept part attends the list as given (an entry listed twice counts
twice), as the sparse attention does.  Both forms are exact when every dropped
block's keys equal their mean and equal dense attention when every block is
kept.

Parity: pinned to the mathematics of the expansion (a term-by-term sum over
tokens, exactness cases, second-order convergence in the key deviations, and
the first order of the block-mean form where queries vary); the paper's own
formula is not in its text, so parity against the paper is unpinned.
"""
from __future__ import annotations

import numpy as np

from .blocks import block_bounds, pool_blocks


def block_moments(k: np.ndarray, v: np.ndarray, block: int):
    """Block means and moments of the keys and values.

    k, v : float64 [..., N, D]
    returns (kbar [..., nB, D], vbar [..., nB, D], M [..., nB, D, D]) with
    M[..., j, e, d] = sum over the valid tokens t of block j of
    V[t, e] * (K[t, d] - kbar[j, d]).
    """
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n, d = k.shape[-2], k.shape[-1]
    bounds = block_bounds(n, block)
    kbar = pool_blocks(k, block)
    vbar = pool_blocks(v, block)
    m = np.empty(k.shape[:-2] + (len(bounds), v.shape[-1], d), dtype=np.float64)
    for j, (a, b) in enumerate(bounds):
        dk = k[..., a:b, :] - kbar[..., j:j + 1, :]
        m[..., j, :, :] = np.matmul(np.swapaxes(v[..., a:b, :], -1, -2), dk)
    return kbar, vbar, m


def moment_times_query(mom: np.ndarray, qr: np.ndarray) -> np.ndarray:
    """(M_j q_n)[e] = sum_d M_j[e, d] q_n[d] for every query n and block j.

    mom : [J, D, D]; qr : [n, D]  ->  [n, J, D]
    """
    return np.einsum("jed,nd->nje", mom, qr)


def log_token_count(count: np.ndarray) -> np.ndarray:
    """ln n_j: a dropped block stands for its n_j tokens in the zero-order sum."""
    return np.log(count)


def dropped_blocks(kept_row, n_blocks: int):
    """Blocks of [0, nB) that no in-range entry of the row's list names."""
    named = {int(j) for j in kept_row if 0 <= int(j) < n_blocks}
    return [j for j in range(n_blocks) if j not in named]


def first_order_log_weights(qr: np.ndarray, qbar_i: np.ndarray, kbar_drop: np.ndarray, scale: float,
                            weight: str) -> np.ndarray:
    """Natural-log weights of the first-order terms, [n, J]: c q_n.kbar_j for
    the plain expansion (weight="query"), c qbar_i.kbar_j for every query of
    the block in the block-mean form (weight="block_mean")."""
    if weight == "query":
        return scale * (qr @ kbar_drop.T)
    if weight == "block_mean":
        return np.broadcast_to(scale * (qbar_i @ kbar_drop.T), (qr.shape[0], kbar_drop.shape[0]))
    raise ValueError(f"weight must be 'query' or 'block_mean', not {weight!r}")


def remainder_attention(q, k, v, kept, block: int, scale: float, rows=None, first_order: bool = True,
                        weight: str = "query"):
    """Attention over the kept blocks plus the first-order remainder of the
    dropped ones (the definition in the module docstring).

    q, k, v     : float64 [B, H, N, D]
    kept        : kept[b][h][i] = iterable of KV block indices
    rows        : optional iterable of (b, h, i); other query blocks stay NaN
    first_order : False leaves out the c M_j q terms (zero order only), which
                  gives the size of the first-order part as a difference
    weight      : "query" (the plain expansion) or "block_mean" (the block-mean
                  query in the first-order weight, as the GPU kernels compute)
    returns (out float64 [B, H, N, D], lse float64 [B, H, N])
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, H, N, D = q.shape
    bounds = block_bounds(N, block)
    nb = len(bounds)
    qbar = pool_blocks(q, block)
    kbar, vbar, mom = block_moments(k, v, block)
    count = np.array([b - a for a, b in bounds], dtype=np.float64)
    out = np.full((B, H, N, D), np.nan)
    lse = np.full((B, H, N), np.nan)
    if rows is None:
        rows = [(b, h, i) for b in range(B) for h in range(H) for i in range(nb)]
    for b, h, i in rows:
        qa, qb = bounds[i]
        listed = [int(j) for j in kept[b][h][i] if 0 <= int(j) < nb]
        drop = dropped_blocks(listed, nb)
        key_tok = (np.concatenate([np.arange(*bounds[j]) for j in listed])
                   if listed else np.zeros(0, dtype=np.int64))
        qr = q[b, h, qa:qb]                                   # [n, D]
        # exponents (natural log) of every term, then one common reference
        a_log = scale * (qr @ k[b, h, key_tok].T)              # kept keys     [n, m]
        z_log = scale * (qr @ kbar[b, h, drop].T) + log_token_count(count[drop])   # zero order [n, J]
        f_log = first_order_log_weights(qr, qbar[b, h, i], kbar[b, h, drop], scale, weight)   # [n, J]
        ref = np.max(np.concatenate([a_log, z_log, f_log], axis=1), axis=1, keepdims=True)
        wa = np.exp(a_log - ref)
        wz = np.exp(z_log - ref)
        wf = np.exp(f_log - ref)
        den = wa.sum(axis=1) + wz.sum(axis=1)
        num = wa @ v[b, h, key_tok] + wz @ vbar[b, h, drop]
        # first-order values: sum_j wf[n, j] * c * M_j q_n
        if first_order:
            mq = moment_times_query(mom[b, h, drop], qr)       # [n, J, D]
            num = num + scale * np.einsum("nj,nje->ne", wf, mq)
        out[b, h, qa:qb] = num / den[:, None]
        lse[b, h, qa:qb] = ref[:, 0] + np.log(den)
    return out, lse
