"""Pins for the oracle's bf16 decoding, block partition and block pooling.

Nothing here calls the oracle twice to check itself: expectations come from
closed forms (IEEE bf16 bit patterns, arithmetic-progression means) and from a
pure-Python brute force written independently of the numpy code.
"""
import math

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.cpu


def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0001, 0x7F7F, 0x8000, 0x4049], dtype=np.uint16)
    want = [1.0, -2.0, 1.0 + 2.0 ** -7, 2.0 ** -133, (2 - 2.0 ** -7) * 2.0 ** 127, -0.0, 3.140625]
    got = oracle.bf16_bits_to_f64(bits)
    assert got.dtype == np.float64
    for g, w in zip(got, want):
        assert g == w
    assert math.copysign(1.0, got[5]) == -1.0


@pytest.mark.parametrize("n,s", [(1024, 64), (1000, 64), (32760, 64), (63240, 64), (111600, 128),
                                 (75600, 64), (1, 64), (64, 64), (65, 64)])
def test_num_blocks_closed_form(n, s):
    nb = oracle.num_blocks(n, s)
    assert (nb - 1) * s < n <= nb * s
    bounds = oracle.block_bounds(n, s)
    assert len(bounds) == nb
    assert bounds[0][0] == 0 and bounds[-1][1] == n
    assert all(b[1] == c[0] for b, c in zip(bounds, bounds[1:]))
    assert all(b[1] - b[0] == s for b in bounds[:-1])


def test_workload_block_counts():
    # ceil(N/S) and the size of the last block for the five workload shapes
    table = {(1024, 64): (16, 64), (32760, 64): (512, 56), (63240, 64): (989, 8),
             (111600, 128): (872, 112), (75600, 64): (1182, 16)}
    for (n, s), (nb, last) in table.items():
        b = oracle.block_bounds(n, s)
        assert len(b) == nb
        assert b[-1][1] - b[-1][0] == last


def test_pool_arithmetic_progression_closed_form():
    # x[n, d] = n + 1000 d: the mean of tokens a..b-1 is (a + b - 1) / 2 + 1000 d.
    n, s, d = 1000, 64, 5
    x = (np.arange(n)[:, None] + 1000.0 * np.arange(d)[None, :])[None, None]
    p = oracle.pool_blocks(x, s)
    assert p.shape == (1, 1, 16, d)
    for i in range(16):
        a, b = i * s, min((i + 1) * s, n)
        for c in range(d):
            assert p[0, 0, i, c] == (a + b - 1) / 2.0 + 1000.0 * c
    # last block has 40 tokens (960..999): its mean is 979.5, not the zero-padded 612.1875
    assert p[0, 0, 15, 0] == 979.5


def test_pool_bruteforce_pure_python():
    rng = np.random.default_rng(3)
    B, H, N, D, S = 2, 3, 37, 4, 8
    x = rng.standard_normal((B, H, N, D))
    p = oracle.pool_blocks(x, S)
    for b in range(B):
        for h in range(H):
            for i in range(5):
                toks = [t for t in range(N) if t // S == i]
                for c in range(D):
                    want = math.fsum(float(x[b, h, t, c]) for t in toks) / len(toks)
                    assert abs(p[b, h, i, c] - want) <= 1e-14 * (1 + abs(want))


def test_pool_keeps_heads_separate():
    # a per-head constant must pool to itself: catches mixing of the head axis with tokens
    B, H, N, D, S = 1, 4, 130, 2, 64
    x = np.broadcast_to(np.arange(H, dtype=np.float64)[None, :, None, None], (B, H, N, D)).copy()
    p = oracle.pool_blocks(x, S)
    assert np.all(p == np.arange(H)[None, :, None, None])


def test_pool_golden_partial_block(golden_dir):
    import json, os
    g = json.load(open(os.path.join(golden_dir, "select_handworked.json")))["pool_topk"]
    k = np.array(g["k_tokens"], dtype=np.float64)[None, None]
    q = np.array(g["q_tokens"], dtype=np.float64)[None, None]
    kp = oracle.pool_blocks(k, g["block"])[0, 0]
    qp = oracle.pool_blocks(q, g["block"])[0, 0]
    assert kp.tolist() == [[2, 0], [0, 2], [1, 1], [-1, 1.5]]
    assert qp.tolist() == [[1, 0], [0, 2], [1, 1], [0, 1]]
