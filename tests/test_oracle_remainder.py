"""Pins of the oracle's first-order remainder for dropped key blocks.

What the mathematics fixes for the plain expansion of each dropped key's
exponential about its block's mean key (Section 4.2.2's first-order
compensation), and for the block-mean-query form the GPU kernels compute:
  - the moments by brute force over tokens, and by an independent identity;
  - the plain expansion summed term by term over the dropped tokens, with no
    moments: exp(c q.kbar_j) (1 + c q.(k_t - kbar_j)) as the weight of V[t];
  - exactness when every key of a block equals the block mean (the result is
    then plain dense attention, LSE included), in both forms;
  - every block kept: plain dense attention; constant values: that value;
  - with queries and keys both close to their block means, the error against
    dense attention is second order (halving the deviations divides it by
    about four) in both forms, which a dropped, transposed or mis-signed
    first-order term would turn into first order;
  - with queries that differ by order one inside a block and keys close to
    their means, the plain expansion is still second order in the key
    deviation while the block-mean form is first order (halving divides its
    error by about two): this tells the two forms apart.
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


def test_first_order_term_by_term():
    """The plain expansion as a sum over the dropped tokens themselves: every
    dropped key t of block j contributes weight w = exp(c q.kbar_j) (1 + c
    q.(k_t - kbar_j)) and value w V[t]; the kept keys their exact weights."""
    rng = np.random.default_rng(41)
    N, S, D, c = 22, 5, 3, 0.6                            # blocks of 5, 5, 5, 5, 2 tokens
    q, k, v = (rng.standard_normal((1, 1, N, D)) for _ in range(3))
    nb = 5
    bounds = [(0, 5), (5, 10), (10, 15), (15, 20), (20, 22)]
    kept = [[[[1], [], [0, 4], [3, 2, 1, 0, 4], [2]]]]
    out, lse = orem.remainder_attention(q, k, v, kept, S, c)
    for i in range(nb):
        listed = kept[0][0][i]
        for n in range(*bounds[i]):
            qn = q[0, 0, n]
            den = 0.0
            num = np.zeros(D)
            for j, (a, b) in enumerate(bounds):
                kb = sum(k[0, 0, t] for t in range(a, b)) / (b - a)
                for t in range(a, b):
                    if j in listed:
                        w = np.exp(c * float(qn @ k[0, 0, t]))
                    else:
                        w = np.exp(c * float(qn @ kb)) * (1.0 + c * float(qn @ (k[0, 0, t] - kb)))
                    den += w
                    num += w * v[0, 0, t]
            assert np.abs(out[0, 0, n] - num / den).max() < 1e-12, (i, n)
            assert abs(lse[0, 0, n] - np.log(den)) < 1e-12, (i, n)


WEIGHTS = ["query", "block_mean"]


@pytest.mark.parametrize("weight", WEIGHTS)
@pytest.mark.parametrize("N,S", [(37, 8), (40, 8), (9, 4)])
def test_constant_key_blocks_equal_dense(N, S, weight):
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
    out, lse = orem.remainder_attention(q, k, v, [kept], S, 0.4, weight=weight)
    ref, rlse = oracle.dense_attention(q, k, v, 0.4, block=S)
    assert np.abs(out - ref).max() < 1e-12
    assert np.abs(lse - rlse).max() < 1e-12


@pytest.mark.parametrize("weight", WEIGHTS)
def test_keep_all_equals_dense(weight):
    rng = np.random.default_rng(8)
    N, S, D = 29, 8, 5
    nb = 4
    q, k, v = (rng.standard_normal((1, 1, N, D)) for _ in range(3))
    kept = [[[list(range(nb)) for _ in range(nb)]]]
    out, lse = orem.remainder_attention(q, k, v, kept, S, 0.5, weight=weight)
    ref, rlse = oracle.dense_attention(q, k, v, 0.5, block=S)
    assert np.abs(out - ref).max() < 1e-12
    assert np.abs(lse - rlse).max() < 1e-12


@pytest.mark.parametrize("weight", WEIGHTS)
def test_constant_values_give_the_value(weight):
    rng = np.random.default_rng(9)
    N, S, D = 45, 8, 6
    nb = 6
    q, k = (rng.standard_normal((1, 1, N, D)) for _ in range(2))
    v0 = rng.standard_normal(D)
    v = np.broadcast_to(v0, (1, 1, N, D)).copy()
    kept = [[[[i] if i % 2 else [] for i in range(nb)]]]
    out, _ = orem.remainder_attention(q, k, v, kept, S, 0.5, weight=weight)
    assert np.abs(out[0, 0] - v0).max() < 1e-12


def _deviation_case(eps, vary_queries=True, seed=1, N=40, S=8, D=16, query_spread=None):
    """Blocks of S tokens, each row keeping only its own block; keys deviate
    from their block means by eps.  Queries deviate by eps too (vary_queries),
    not at all, or by the fixed amount query_spread (order one)."""
    rng = np.random.default_rng(seed)
    nb = N // S
    qb = 0.7 * rng.standard_normal((nb, D))
    kb = 0.7 * rng.standard_normal((nb, D))
    a = rng.standard_normal((N, D)) if vary_queries else np.zeros((N, D))
    u = rng.standard_normal((N, D))
    v = rng.standard_normal((1, 1, N, D))
    qdev = eps * a if query_spread is None else query_spread * rng.standard_normal((N, D))
    q = (np.repeat(qb, S, axis=0) + qdev)[None, None]
    k = (np.repeat(kb, S, axis=0) + eps * u)[None, None]
    kept = [[[[i] for i in range(nb)]]]                  # each row keeps its own block
    return q, k, v, kept, S


@pytest.mark.parametrize("weight", WEIGHTS)
@pytest.mark.parametrize("vary_queries", [True, False], ids=["queries_and_keys", "keys_only"])
def test_error_is_second_order(vary_queries, weight):
    errs = []
    for eps in (0.02, 0.01, 0.005):
        q, k, v, kept, S = _deviation_case(eps, vary_queries)
        out, _ = orem.remainder_attention(q, k, v, kept, S, 0.25, weight=weight)
        ref, _ = oracle.dense_attention(q, k, v, 0.25, block=S)
        errs.append(np.abs(out - ref).max())
    ratios = [errs[0] / errs[1], errs[1] / errs[2]]
    assert all(3.6 < r < 4.4 for r in ratios), (errs, ratios)
    # and the remainder is what makes it small: dropping the blocks is off by O(1)
    q, k, v, kept, S = _deviation_case(0.005, vary_queries)
    sparse, _ = oracle.block_sparse_attention(q, k, v, kept, S, 0.25)
    ref, _ = oracle.dense_attention(q, k, v, 0.25, block=S)
    assert np.abs(sparse - ref).max() > 1000 * errs[-1]


def _key_deviation_errors(weight):
    errs = []
    for eps in (0.02, 0.01, 0.005):
        q, k, v, kept, S = _deviation_case(eps, query_spread=1.0, seed=3)
        out, _ = orem.remainder_attention(q, k, v, kept, S, 0.25, weight=weight)
        ref, _ = oracle.dense_attention(q, k, v, 0.25, block=S)
        errs.append(np.abs(out - ref).max())
    return errs, [errs[0] / errs[1], errs[1] / errs[2]]


def test_plain_expansion_is_second_order_in_the_key_deviation():
    """Queries spread by order one inside each block, keys by eps: the plain
    expansion's error against dense attention falls fourfold per halving."""
    errs, ratios = _key_deviation_errors("query")
    assert all(3.6 < r < 4.4 for r in ratios), (errs, ratios)


def test_block_mean_form_is_first_order_in_the_key_deviation():
    """The same cases through the block-mean form: its first-order weight is
    off by an order-one factor for queries away from the block mean, so the
    error falls only twofold per halving, and is far above the plain one."""
    errs, ratios = _key_deviation_errors("block_mean")
    assert all(1.8 < r < 2.2 for r in ratios), (errs, ratios)
    plain, _ = _key_deviation_errors("query")
    assert errs[-1] > 20 * plain[-1], (errs, plain)


def test_forms_share_the_denominator():
    """The block-mean form changes only the first-order numerator, so both
    forms give the same LSE."""
    q, k, v, kept, S = _deviation_case(0.3, query_spread=1.0, seed=4)
    _, l1 = orem.remainder_attention(q, k, v, kept, S, 0.25, weight="query")
    _, l2 = orem.remainder_attention(q, k, v, kept, S, 0.25, weight="block_mean")
    assert np.abs(l1 - l2).max() < 1e-12
