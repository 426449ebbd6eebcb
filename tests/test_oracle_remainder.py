"""Pins of the oracle's first-order remainder for dropped key blocks.

What the mathematics fixes for the reading (expansion of each dropped block's
exponentials about the block means, Section 4.2.2's first-order compensation):
  - the moments by brute force over tokens, and by an independent identity;
  - exactness when every key of a block equals the block mean (the result is
    then plain dense attention, LSE included);
  - every block kept: plain dense attention;
  - constant values: the output is that value;
  - the error against dense attention is second order in the query and key
    deviations (halving them divides it by about four), which a dropped,
    transposed or mis-signed first-order term would turn into first order.
"""
import numpy as np
import pytest

import oracle
import oracle.remainder as orem

pytestmark = pytest.mark.cpu


def test_moments_bruteforce_and_identity():
    rng = np.random.default_rng(31)
    N, D, S = 11, 3, 4                                   # blocks of 4, 4, 3 tokens
    k = rng.standard_normal((1, 2, N, D))
    v = rng.standard_normal((1, 2, N, D))
    kbar, vbar, mom = orem.block_moments(k, v, S)
    bounds = [(0, 4), (4, 8), (8, 11)]
    for h in range(2):
        for j, (a, b) in enumerate(bounds):
            n = b - a
            km = [sum(k[0, h, t, d] for t in range(a, b)) / n for d in range(D)]
            vm = [sum(v[0, h, t, e] for t in range(a, b)) / n for e in range(D)]
            assert np.allclose(kbar[0, h, j], km, rtol=0, atol=1e-14)
            assert np.allclose(vbar[0, h, j], vm, rtol=0, atol=1e-14)
            for e in range(D):
                for d in range(D):
                    want = sum(v[0, h, t, e] * (k[0, h, t, d] - km[d]) for t in range(a, b))
                    assert abs(mom[0, h, j, e, d] - want) < 1e-13, (h, j, e, d)
            # sum_t v_t (k_t - kbar)^T = V^T K - n vbar kbar^T
            ident = v[0, h, a:b].T @ k[0, h, a:b] - n * np.outer(vbar[0, h, j], kbar[0, h, j])
            assert np.allclose(mom[0, h, j], ident, rtol=0, atol=1e-13)


def _constant_key_case(seed, N, S, D):
    rng = np.random.default_rng(seed)
    nb = -(-N // S)
    q = rng.standard_normal((1, 2, N, D))
    v = rng.standard_normal((1, 2, N, D))
    kb = rng.standard_normal((1, 2, nb, D))
    k = np.repeat(kb, S, axis=2)[:, :, :N]               # every key equals its block mean
    return q, k, v, nb, rng


@pytest.mark.parametrize("N,S", [(37, 8), (40, 8), (9, 4)])
def test_constant_key_blocks_equal_dense(N, S):
    q, k, v, nb, rng = _constant_key_case(5 + N, N, S, 6)
    kept = [[[] for _ in range(nb)] for _ in range(2)]
    for h in range(2):
        for i in range(nb):
            kind = (i + h) % 4
            if kind == 0:
                kept[h][i] = []                                   # nothing kept
            elif kind == 1:
                kept[h][i] = list(range(nb))                      # everything kept
            elif kind == 2:
                kept[h][i] = sorted(rng.choice(nb, size=max(1, nb // 3), replace=False).tolist())
            else:
                kept[h][i] = [nb - 1, -1, nb + 2, 0]              # ragged block, out-of-range entries
    out, lse = orem.remainder_attention(q, k, v, [kept], S, 0.4)
    ref, rlse = oracle.dense_attention(q, k, v, 0.4, block=S)
    assert np.abs(out - ref).max() < 1e-12
    assert np.abs(lse - rlse).max() < 1e-12


def test_keep_all_equals_dense():
    rng = np.random.default_rng(8)
    N, S, D = 29, 8, 5
    nb = 4
    q, k, v = (rng.standard_normal((1, 1, N, D)) for _ in range(3))
    kept = [[[list(range(nb)) for _ in range(nb)]]]
    out, lse = orem.remainder_attention(q, k, v, kept, S, 0.5)
    ref, rlse = oracle.dense_attention(q, k, v, 0.5, block=S)
    assert np.abs(out - ref).max() < 1e-12
    assert np.abs(lse - rlse).max() < 1e-12


def test_constant_values_give_the_value():
    rng = np.random.default_rng(9)
    N, S, D = 45, 8, 6
    nb = 6
    q, k = (rng.standard_normal((1, 1, N, D)) for _ in range(2))
    v0 = rng.standard_normal(D)
    v = np.broadcast_to(v0, (1, 1, N, D)).copy()
    kept = [[[[i] if i % 2 else [] for i in range(nb)]]]
    out, _ = orem.remainder_attention(q, k, v, kept, S, 0.5)
    assert np.abs(out[0, 0] - v0).max() < 1e-12


def _deviation_case(eps, vary_queries=True, seed=1, N=40, S=8, D=16):
    rng = np.random.default_rng(seed)
    nb = N // S
    qb = 0.7 * rng.standard_normal((nb, D))
    kb = 0.7 * rng.standard_normal((nb, D))
    a = rng.standard_normal((N, D)) if vary_queries else np.zeros((N, D))
    u = rng.standard_normal((N, D))
    v = rng.standard_normal((1, 1, N, D))
    q = (np.repeat(qb, S, axis=0) + eps * a)[None, None]
    k = (np.repeat(kb, S, axis=0) + eps * u)[None, None]
    kept = [[[[i] for i in range(nb)]]]                  # each row keeps its own block
    return q, k, v, kept, S


@pytest.mark.parametrize("vary_queries", [True, False], ids=["queries_and_keys", "keys_only"])
def test_error_is_second_order(vary_queries):
    errs = []
    for eps in (0.02, 0.01, 0.005):
        q, k, v, kept, S = _deviation_case(eps, vary_queries)
        out, _ = orem.remainder_attention(q, k, v, kept, S, 0.25)
        ref, _ = oracle.dense_attention(q, k, v, 0.25, block=S)
        errs.append(np.abs(out - ref).max())
    ratios = [errs[0] / errs[1], errs[1] / errs[2]]
    assert all(3.6 < r < 4.4 for r in ratios), (errs, ratios)
    # and the remainder is what makes it small: dropping the blocks is off by O(1)
    q, k, v, kept, S = _deviation_case(0.005, vary_queries)
    sparse, _ = oracle.block_sparse_attention(q, k, v, kept, S, 0.25)
    ref, _ = oracle.dense_attention(q, k, v, 0.25, block=S)
    assert np.abs(sparse - ref).max() > 1000 * errs[-1]
