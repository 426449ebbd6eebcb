"""Pins of the token-pruning oracle: a library norm, closed forms, a
pure-Python sort with an explicit tie key, exact ties, a hand-worked example,
and gather/scatter identities."""
import math

import numpy as np
import pytest

import oracle.token_prune as otp

pytestmark = pytest.mark.cpu


def test_scores_are_squared_library_norms_and_closed_form():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((2, 7, 33))
    assert np.allclose(otp.token_scores(x), np.linalg.norm(x, axis=-1) ** 2, rtol=1e-13)
    c = np.full((1, 3, 10), 2.5)
    c[0, 1] = -1.0
    assert np.array_equal(otp.token_scores(c), [[62.5, 10.0, 62.5]])
    # the channel axis, not the token axis: a transposed reduction gives other numbers
    y = np.zeros((1, 2, 3))
    y[0, 0] = [1.0, 2.0, 2.0]
    assert np.array_equal(otp.token_scores(y), [[9.0, 0.0]])


def test_keep_count():
    assert otp.keep_count(111600, 0.5) == 55800
    assert otp.keep_count(10, 0.25) == 3          # ceil(2.5)
    assert otp.keep_count(1180, 0.1) == 118       # 0.1 * 1180 = 118.00000000000001
    assert otp.keep_count(7, 1e-9) == 1
    assert otp.keep_count(7, 1.0) == 7


def test_select_matches_python_sort_with_ties():
    rng = np.random.default_rng(2)
    s = rng.integers(0, 6, size=(3, 40)).astype(np.float64)      # many exact ties
    for k in (1, 7, 20, 40):
        got = otp.select_tokens(s, k)
        for b in range(3):
            want = sorted(sorted(range(40), key=lambda n: (-s[b, n], n))[:k])
            assert got[b].tolist() == want


def test_select_hand_worked():
    s = np.array([[3.0, 9.0, 1.0, 9.0, 4.0, 3.0]])
    # best three: 9 (token 1), 9 (token 3), 4 (token 4); of the 3s neither is needed
    assert otp.select_tokens(s, 3).tolist() == [[1, 3, 4]]
    # best four: the tie at 3 goes to the lower index (token 0)
    assert otp.select_tokens(s, 4).tolist() == [[0, 1, 3, 4]]


def test_gather_scatter_identities():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 9, 4))
    kept = np.array([[0, 2, 5, 8], [1, 3, 4, 7]])
    g = otp.gather_tokens(x, kept)
    assert g.shape == (2, 4, 4)
    assert np.array_equal(g[1, 2], x[1, 4])
    # putting the gathered rows back over the input returns the input
    assert np.array_equal(otp.scatter_tokens(g, kept, x), x)
    # processed rows land at their positions, dropped rows keep the base
    out = otp.scatter_tokens(np.zeros_like(g), kept, x)
    assert np.all(out[0, [0, 2, 5, 8]] == 0) and np.array_equal(out[0, [1, 3, 4, 6, 7]], x[0, [1, 3, 4, 6, 7]])
    assert np.array_equal(out[1, [0, 2, 5, 6, 8]], x[1, [0, 2, 5, 6, 8]])
