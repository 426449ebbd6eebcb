"""Pins of the QKNorm + RoPE + pool oracle against things other than itself:
bit-level bf16 rounding, closed forms of RMSNorm, a library norm, RoPE as
complex multiplication (cmath), hand-derived angles, and the invariants of a
rotation (identity at the origin, norm preservation, relative position)."""
import cmath
import math

import numpy as np
import pytest

import oracle.qknorm_rope as oqr

pytestmark = pytest.mark.cpu


def _bf16_from_f32_bits(x32: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> bf16 on the bit pattern (the usual
    integer trick), back to float64."""
    b = np.asarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return (r.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def test_round_bf16_matches_bit_level_rounding_on_float32_values():
    rng = np.random.default_rng(7)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32),
                        (rng.standard_normal(2000) * 1e-30).astype(np.float32),
                        (rng.standard_normal(2000) * 1e30).astype(np.float32)])
    assert np.array_equal(oqr.round_bf16(x.astype(np.float64)), _bf16_from_f32_bits(x))


def test_round_bf16_ties_and_no_double_rounding():
    # bf16 spacing at 1 is 2^-7; 1 + 2^-8 is a tie between 1 (even) and 1 + 2^-7
    assert oqr.round_bf16(np.array([1 + 2 ** -8]))[0] == 1.0
    assert oqr.round_bf16(np.array([1 + 3 * 2 ** -8]))[0] == 1 + 2 ** -6
    assert oqr.round_bf16(np.array([-(1 + 2 ** -8)]))[0] == -1.0
    # just above the tie: must round up, although float32 would first round it
    # onto the tie (a double rounding that would give 1.0)
    x = 1 + 2 ** -8 + 2 ** -30
    assert np.float32(x) == np.float32(1 + 2 ** -8)
    assert oqr.round_bf16(np.array([x]))[0] == 1 + 2 ** -7
    # already representable values stay
    for v in (0.0, 1.0, -3.25, 2.0 ** -126, 1.5 * 2 ** 100):
        assert oqr.round_bf16(np.array([v]))[0] == v


def test_rms_norm_closed_forms():
    D = 8
    for c, eps in ((3.0, 0.0), (0.5, 1e-2), (-2.0, 1e-6)):
        x = np.full(D, c)
        gamma = np.arange(1.0, D + 1)
        y = oqr.rms_norm(x, gamma, eps)
        assert np.allclose(y, c / math.sqrt(c * c + eps) * gamma, rtol=1e-14, atol=0)
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 128))
    # eps = 0, gamma = 1: x scaled to unit RMS, i.e. x * sqrt(D) / ||x||
    y = oqr.rms_norm(x, np.ones(128), 0.0)
    assert np.allclose(y, x * math.sqrt(128) / np.linalg.norm(x, axis=-1, keepdims=True), rtol=1e-13)
    assert np.allclose(oqr.rms_norm(7.0 * x, np.ones(128), 0.0), y, rtol=1e-13)


def test_rope_pair_groups():
    assert oqr.rope_pair_groups(128) == (22, 21, 21)
    assert oqr.rope_pair_groups(112) == (20, 18, 18)
    assert oqr.rope_pair_groups(64) == (12, 10, 10)
    assert oqr.rope_pair_groups(6) == (1, 1, 1)


def test_rope_angles_hand_derived():
    # D = 12: pairs 0,1 follow t, 2,3 follow y, 4,5 follow x; base 100 gives
    # frequencies 100^0 = 1 and 100^(-1/2) = 0.1 in every group
    grid = (4, 3, 6)
    ang = oqr.rope_angles(grid, 12, 100.0)
    n = (3 * 3 + 2) * 6 + 5                        # token (t, y, x) = (3, 2, 5)
    assert np.allclose(ang[n], [3.0, 0.3, 2.0, 0.2, 5.0, 0.5], rtol=1e-15, atol=1e-15)
    assert np.all(ang[0] == 0.0)                    # the origin


def test_rope_is_complex_multiplication():
    rng = np.random.default_rng(3)
    grid = (3, 4, 5)
    D = 12
    N = grid[0] * grid[1] * grid[2]
    x = rng.standard_normal((N, D))
    ang = oqr.rope_angles(grid, D, 100.0)
    y = oqr.apply_rope(x, ang)
    for n in (0, 7, N - 1):
        for p in range(D // 2):
            z = complex(x[n, 2 * p], x[n, 2 * p + 1]) * cmath.exp(1j * ang[n, p])
            assert abs(complex(y[n, 2 * p], y[n, 2 * p + 1]) - z) < 1e-12


def test_rope_identity_at_origin_and_norm_preserving():
    rng = np.random.default_rng(4)
    grid = (2, 3, 4)
    x = rng.standard_normal((1, 1, 24, 128))
    y = oqr.apply_rope(x, oqr.rope_angles(grid, 128, 10000.0))
    assert np.array_equal(y[..., 0, :], x[..., 0, :])
    pair_norm = lambda v: v[..., 0::2] ** 2 + v[..., 1::2] ** 2   # noqa: E731
    assert np.allclose(pair_norm(y), pair_norm(x), rtol=1e-12)


def test_rope_relative_position():
    # <R(p1) q, R(p2) k> depends only on p1 - p2 (here: a shift along x, then along t)
    rng = np.random.default_rng(5)
    grid = (4, 3, 8)
    D = 64
    ang = oqr.rope_angles(grid, D, 10000.0)
    q = rng.standard_normal(D)
    k = rng.standard_normal(D)
    tok = lambda t, y, x: (t * grid[1] + y) * grid[2] + x    # noqa: E731

    def dot(a, b):
        return float(oqr.apply_rope(q[None], ang[[a]])[0] @ oqr.apply_rope(k[None], ang[[b]])[0])

    base = dot(tok(1, 1, 2), tok(1, 2, 5))
    assert abs(dot(tok(1, 1, 4), tok(1, 2, 7)) - base) < 1e-10
    assert abs(dot(tok(3, 1, 2), tok(3, 2, 5)) - base) < 1e-10
    assert abs(dot(tok(1, 1, 3), tok(1, 2, 5)) - base) > 1e-6     # a different offset differs


def test_producer_pools_its_rounded_outputs():
    rng = np.random.default_rng(6)
    grid = (2, 3, 10)                                # N = 60: blocks of 16, last one partial
    q = rng.standard_normal((1, 2, 60, 64))
    k = rng.standard_normal((1, 2, 60, 64))
    gq, gk = rng.uniform(0.5, 1.5, 64), rng.uniform(0.5, 1.5, 64)
    qo, ko, qp, kp = oqr.qknorm_rope_pool(q, k, gq, gk, grid, 16, 1e-6, 10000.0)
    assert np.array_equal(oqr.round_bf16(qo), qo) and np.array_equal(oqr.round_bf16(ko), ko)
    for out, pooled in ((qo, qp), (ko, kp)):
        assert pooled.shape == (1, 2, 4, 64)
        assert np.allclose(pooled[..., 1, :], out[..., 16:32, :].mean(axis=-2), rtol=0, atol=1e-15)
        assert np.allclose(pooled[..., 3, :], out[..., 48:60, :].mean(axis=-2), rtol=0, atol=1e-15)
    # and the unrounded values are RMSNorm then RoPE
    exact = oqr.norm_rope(q, gq, grid, 1e-6, 10000.0)
    assert np.max(np.abs(qo - exact) / np.maximum(np.abs(exact), 1e-30)) <= 2.0 ** -8
