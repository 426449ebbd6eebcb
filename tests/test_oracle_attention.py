"""Pins for the oracle's block-sparse and dense attention.

Independent references: pure-Python loops with math.exp/math.fsum on tiny
inputs, torch's scaled_dot_product_attention in float64 on the CPU (a library
routine), closed forms (constant values, block-constant keys/values, one-hot
values exposing the probability rows), and invariants.
"""
import math

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.cpu


def _rand_qkv(rng, B, H, N, D, spread=1.0):
    return tuple(spread * rng.standard_normal((B, H, N, D)) for _ in range(3))


def _all_blocks(B, H, nb):
    return [[[list(range(nb)) for _ in range(nb)] for _ in range(H)] for _ in range(B)]


def _brute_row(q, K, V, keys, c):
    logits = [c * math.fsum(q[d] * K[m][d] for d in range(len(q))) for m in keys]
    mx = max(logits)
    w = [math.exp(l - mx) for l in logits]
    z = math.fsum(w)
    out = [math.fsum(w[a] * V[m][d] for a, m in enumerate(keys)) / z for d in range(len(V[0]))]
    return out, mx + math.log(z)


def test_sparse_bruteforce_pure_python():
    rng = np.random.default_rng(21)
    B, H, N, D, S = 1, 2, 21, 3, 4            # 6 blocks, last holds 1 token
    q, k, v = _rand_qkv(rng, B, H, N, D, 1.5)
    nb = oracle.num_blocks(N, S)
    kept = [[[sorted(rng.choice(nb, size=int(rng.integers(1, nb + 1)), replace=False).tolist())
              for _ in range(nb)] for _ in range(H)]]
    c = 0.7
    out, lse = oracle.block_sparse_attention(q, k, v, kept, S, c)
    for h in range(H):
        for n in range(N):
            i = n // S
            keys = [m for j in kept[0][h][i] for m in range(j * S, min((j + 1) * S, N))]
            o, l = _brute_row(q[0, h, n], k[0, h], v[0, h], keys, c)
            assert np.allclose(out[0, h, n], o, rtol=0, atol=1e-13)
            assert abs(lse[0, h, n] - l) < 1e-13


def test_dense_matches_torch_sdpa_float64():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(22)
    B, H, N, D = 2, 2, 100, 16
    q, k, v = _rand_qkv(rng, B, H, N, D)
    c = 1.0 / math.sqrt(D)
    out, lse = oracle.dense_attention(q, k, v, c, block=32)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), scale=c).numpy()
    assert np.allclose(out, ref, rtol=0, atol=1e-12)
    from scipy.special import logsumexp
    ref_lse = logsumexp(c * np.einsum("bhnd,bhmd->bhnm", q, k), axis=-1)
    assert np.allclose(lse, ref_lse, rtol=0, atol=1e-12)


def test_keep_all_equals_dense():
    rng = np.random.default_rng(23)
    B, H, N, D, S = 1, 2, 150, 8, 32
    q, k, v = _rand_qkv(rng, B, H, N, D)
    nb = oracle.num_blocks(N, S)
    c = 0.3
    o1, l1 = oracle.block_sparse_attention(q, k, v, _all_blocks(B, H, nb), S, c)
    o2, l2 = oracle.dense_attention(q, k, v, c, block=S)
    assert np.allclose(o1, o2, rtol=0, atol=1e-13)
    assert np.allclose(l1, l2, rtol=0, atol=1e-13)


def test_constant_values_give_constant_output():
    rng = np.random.default_rng(24)
    B, H, N, D, S = 1, 1, 70, 4, 16
    q, k, _ = _rand_qkv(rng, B, H, N, D, 3.0)
    v = np.ones((B, H, N, D))
    nb = oracle.num_blocks(N, S)
    kept = [[[[0, nb - 1], [2], [1, 3], [4], [0, 1, 2, 3, 4]]]]
    out, _ = oracle.block_sparse_attention(q, k, v, kept, S, 1.0)
    assert np.allclose(out, 1.0, rtol=0, atol=1e-14)


def test_onehot_values_expose_probability_rows():
    # V = identity over tokens (N <= D) makes O[n] the probability row of query n:
    # non-negative, zero off the kept keys, summing to one, equal to exp(logit - LSE).
    rng = np.random.default_rng(25)
    B, H, N, S = 1, 1, 24, 8
    D = N
    q = rng.standard_normal((B, H, N, 5))
    k = rng.standard_normal((B, H, N, 5))
    v = np.eye(N)[None, None]
    qd = np.zeros((B, H, N, D)); qd[..., :5] = q
    kd = np.zeros((B, H, N, D)); kd[..., :5] = k
    kept = [[[[1], [0, 2], [0, 1, 2]]]]
    c = 0.9
    out, lse = oracle.block_sparse_attention(qd, kd, v, kept, S, c)
    for n in range(N):
        keys = [m for j in kept[0][0][n // S] for m in range(j * S, (j + 1) * S)]
        row = out[0, 0, n]
        assert np.all(row >= 0)
        assert abs(row.sum() - 1.0) < 1e-12
        assert np.all(row[[m for m in range(N) if m not in keys]] == 0)
        for m in keys:
            want = math.exp(c * float(q[0, 0, n] @ k[0, 0, m]) - lse[0, 0, n])
            assert abs(row[m] - want) < 1e-12


def test_block_constant_keys_values_closed_form():
    # K and V constant within each block (kappa_j, nu_j); block j has n_j valid tokens.
    # Then O[n] = sum_j n_j e^{c q.kappa_j} nu_j / sum_j n_j e^{c q.kappa_j}.
    rng = np.random.default_rng(26)
    B, H, N, D, S = 1, 1, 45, 3, 16           # blocks of 16, 16, 13 tokens
    nb = 3
    kappa = rng.standard_normal((nb, D))
    nu = rng.standard_normal((nb, D))
    k = np.zeros((B, H, N, D)); v = np.zeros((B, H, N, D))
    for j in range(nb):
        k[0, 0, j * S:(j + 1) * S] = kappa[j]
        v[0, 0, j * S:(j + 1) * S] = nu[j]
    q = rng.standard_normal((B, H, N, D))
    kept = [[[[0, 2], [1, 2], [0, 1, 2]]]]
    c = 0.8
    out, lse = oracle.block_sparse_attention(q, k, v, kept, S, c)
    cnt = [16, 16, 13]
    for n in range(N):
        js = kept[0][0][n // S]
        w = np.array([cnt[j] * math.exp(c * float(q[0, 0, n] @ kappa[j])) for j in js])
        want = (w[:, None] * nu[js]).sum(0) / w.sum()
        assert np.allclose(out[0, 0, n], want, rtol=0, atol=1e-13)
        assert abs(lse[0, 0, n] - math.log(w.sum())) < 1e-12


def test_single_kept_block_is_textbook_attention():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(27)
    B, H, N, D, S = 1, 1, 96, 8, 32
    q, k, v = _rand_qkv(rng, B, H, N, D)
    kept = [[[[2], [0], [1]]]]
    c = 0.5
    out, _ = oracle.block_sparse_attention(q, k, v, kept, S, c)
    for i, j in enumerate([2, 0, 1]):
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q[:, :, i * S:(i + 1) * S]), torch.from_numpy(k[:, :, j * S:(j + 1) * S]),
            torch.from_numpy(v[:, :, j * S:(j + 1) * S]), scale=c).numpy()
        assert np.allclose(out[:, :, i * S:(i + 1) * S], ref, rtol=0, atol=1e-13)


def test_kept_order_does_not_matter_and_rows_subset():
    rng = np.random.default_rng(28)
    B, H, N, D, S = 1, 2, 90, 4, 16
    q, k, v = _rand_qkv(rng, B, H, N, D)
    kept = [[[[0, 3, 5], [1, 2], [5], [0, 1, 2, 3, 4, 5], [4, 2], [3, 0]] for _ in range(H)]]
    rev = [[[list(reversed(r)) for r in hh] for hh in kept[0]]]
    o1, l1 = oracle.block_sparse_attention(q, k, v, kept, S, 0.6)
    o2, l2 = oracle.block_sparse_attention(q, k, v, rev, S, 0.6)
    assert np.allclose(o1, o2, rtol=0, atol=1e-14) and np.allclose(l1, l2, rtol=0, atol=1e-14)
    o3, _ = oracle.block_sparse_attention(q, k, v, kept, S, 0.6, rows=[(0, 1, 4)])
    assert np.array_equal(o3[0, 1, 64:80], o1[0, 1, 64:80])
    assert np.isnan(o3[0, 0]).all()


def test_empty_row_gives_zero_and_minus_inf():
    rng = np.random.default_rng(29)
    q, k, v = _rand_qkv(rng, 1, 1, 32, 4)
    out, lse = oracle.block_sparse_attention(q, k, v, [[[[], [0]]]], 16, 1.0)
    assert np.all(out[0, 0, :16] == 0) and np.all(np.isneginf(lse[0, 0, :16]))


def test_scale_is_applied():
    # doubling the scale equals doubling q
    rng = np.random.default_rng(30)
    q, k, v = _rand_qkv(rng, 1, 1, 40, 4)
    o1, _ = oracle.dense_attention(q, k, v, 2.0, block=8)
    o2, _ = oracle.dense_attention(2.0 * q, k, v, 1.0, block=8)
    assert np.allclose(o1, o2, rtol=0, atol=1e-13)
