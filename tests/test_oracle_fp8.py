"""Pins of the fp8 (e4m3) quantisation oracle and the attention it feeds: the
format's own code table, a library cast, brute-force nearest-value search,
brute-force scale exponents and grouping, error bounds, the softmax
invariance that makes K smoothing harmless, and an exactly representable case
where quantised attention equals plain attention."""
import math
import struct

import numpy as np
import pytest

import oracle
import oracle.fp8_attention as f8

pytestmark = pytest.mark.cpu


def _finite_table():
    vals = {}
    for c in range(256):
        v = f8.e4m3_value(c)
        if v == v:
            vals[c] = v
    return vals


def test_code_table_fixed_points():
    assert f8.e4m3_value(0x38) == 1.0
    assert f8.e4m3_value(0x7E) == 448.0
    assert f8.e4m3_value(0x01) == 2.0 ** -9
    assert f8.e4m3_value(0x08) == 2.0 ** -6
    assert f8.e4m3_value(0x07) == 7 * 2.0 ** -9
    assert math.isnan(f8.e4m3_value(0x7F)) and math.isnan(f8.e4m3_value(0xFF))
    assert f8.e4m3_value(0xB8) == -1.0
    t = _finite_table()
    assert len(t) == 254 and len(set(t.values())) == 253      # +0 and -0 share a value


def _nearest_even(x, table):
    best = None
    for c, v in table.items():
        d = abs(v - x)
        if best is None or d < best[1] or (d == best[1] and (c & 1) == 0 and (best[0] & 1) == 1):
            best = (c, d)
    return table[best[0]]


def test_rounding_matches_brute_force_nearest_even():
    table = _finite_table()
    grid = sorted(set(v for v in table.values()))
    rng = np.random.default_rng(0)
    xs = list(grid)
    xs += [(a + b) / 2 for a, b in zip(grid[:-1], grid[1:])]           # every midpoint
    xs += [np.nextafter((a + b) / 2, b) for a, b in zip(grid[:-1], grid[1:])]
    xs += [np.nextafter((a + b) / 2, a) for a, b in zip(grid[:-1], grid[1:])]
    xs += list(rng.uniform(-448, 448, 300)) + list(rng.standard_normal(300) * 1e-2)
    got = f8.round_e4m3(np.array(xs))
    for x, g in zip(xs, got):
        assert g == _nearest_even(float(x), table), x


def test_rounding_matches_library_cast_from_float32():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.uniform(-448, 448, 20000), rng.standard_normal(20000) * 0.05,
                        rng.standard_normal(5000) * 1e-3]).astype(np.float32)
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(f8.round_e4m3(x.astype(np.float64)), want)


def test_encode_round_trips_every_code():
    t = _finite_table()
    codes = np.array(sorted(t), dtype=np.uint8)
    vals = np.array([t[c] for c in codes])
    vals[codes == 0x80] = -0.0
    assert np.array_equal(f8.encode_e4m3(vals), codes)


def test_scale_exponent_brute_force():
    rng = np.random.default_rng(2)
    cases = [448.0, np.nextafter(448.0, 1e9), 224.0, np.nextafter(224.0, 1e9), 1.0, 3.0e38,
             1e-30, 2.0 ** -140] + list(np.exp(rng.uniform(-60, 60, 400)))
    for a in cases:
        want = next(e for e in range(-127, 128) if a <= 448.0 * 2.0 ** e) if a <= 448.0 * 2.0 ** 127 else 127
        assert f8.scale_exponent(a) == want, a
    assert f8.scale_exponent(0.0) == 0


def test_quantize_error_bounds_and_range():
    rng = np.random.default_rng(3)
    x = rng.standard_normal(5000) * np.exp(rng.uniform(-8, 8, 5000))
    e = f8.scale_exponent(np.abs(x).max())
    y = x * 2.0 ** -e
    assert np.abs(y).max() <= 448.0 and np.abs(y).max() > 224.0      # the scale is tight
    dq = f8.quantize_groups(x, e)
    normal = np.abs(y) >= 2.0 ** -6
    assert np.all(np.abs(dq - x)[normal] <= 2.0 ** -4 * np.abs(x)[normal])
    assert np.all(np.abs(dq - x)[~normal] <= 2.0 ** -10 * 2.0 ** e)


def _bf16(x):
    return oracle.round_bf16(x)


def test_quantize_qkv_matches_pure_python_grouping():
    """Tiny case, element by element: block exponents of Q and smoothed K,
    channel exponents of V, the bf16 channel mean, and every code."""
    rng = np.random.default_rng(4)
    B, H, N, D, S = 1, 2, 10, 4, 4
    q = _bf16(rng.standard_normal((B, H, N, D)) * 3)
    k = _bf16(rng.standard_normal((B, H, N, D)) + 5.0)             # a channel bias to smooth away
    v = _bf16(rng.standard_normal((B, H, N, D)) * np.array([0.1, 1, 10, 100]))
    out = f8.quantize_qkv(q, k, v, S)
    table = _finite_table()
    for h in range(H):
        mean = [float(_bf16(np.array(sum(k[0, h, n, d] for n in range(N)) / N))) for d in range(D)]
        assert np.array_equal(out["k_mean"][0, h], mean)
        ks = [[float(np.float32(k[0, h, n, d]) - np.float32(mean[d])) for d in range(D)] for n in range(N)]
        for i, a in enumerate(range(0, N, S)):
            z = min(N, a + S)
            qa = max(abs(q[0, h, n, d]) for n in range(a, z) for d in range(D))
            ka = max(abs(ks[n][d]) for n in range(a, z) for d in range(D))
            eq = next(e for e in range(-127, 128) if qa <= 448 * 2.0 ** e)
            ek = next(e for e in range(-127, 128) if ka <= 448 * 2.0 ** e)
            assert out["q_exp"][0, h, i] == eq and out["k_exp"][0, h, i] == ek
            for n in range(a, z):
                for d in range(D):
                    assert out["q_code"][0, h, n, d] == _nearest_even(q[0, h, n, d] * 2.0 ** -eq, table)
                    assert out["k_code"][0, h, n, d] == _nearest_even(ks[n][d] * 2.0 ** -ek, table)
        for d in range(D):
            va = max(abs(v[0, h, n, d]) for n in range(N))
            ev = next(e for e in range(-127, 128) if va <= 448 * 2.0 ** e)
            assert out["v_exp"][0, h, d] == ev
            for n in range(N):
                assert out["v_code"][0, h, n, d] == _nearest_even(v[0, h, n, d] * 2.0 ** -ev, table)
    assert np.array_equal(out["q_hat"], np.ldexp(out["q_code"], out["q_exp"][:, :, [0, 0, 0, 0, 1, 1, 1, 1, 2, 2]][..., None]))


def test_smoothing_leaves_attention_unchanged():
    """Adding one vector to every key shifts each query's logits by a
    constant, which the softmax removes."""
    rng = np.random.default_rng(5)
    B, H, N, D, S = 1, 1, 24, 8, 8
    q, k, v = (rng.standard_normal((B, H, N, D)) for _ in range(3))
    kept = [[[[0, 2], [1], [0, 1, 2]]]]
    a, la = oracle.block_sparse_attention(q, k, v, kept, S, 0.3)
    b, lb = oracle.block_sparse_attention(q, k + rng.standard_normal(D) * 4, v, kept, S, 0.3)
    assert np.allclose(a, b, atol=1e-12)


def test_exactly_representable_inputs_lose_nothing():
    """Inputs that are e4m3 values times one power of two per group, with a
    zero K channel mean: quantised attention equals plain attention."""
    rng = np.random.default_rng(6)
    B, H, N, D, S = 1, 2, 32, 8, 8
    grid = np.array([v for v in _finite_table().values() if abs(v) >= 2.0 ** -3])
    q = rng.choice(grid, (B, H, N, D)) * 2.0 ** -4
    half = rng.choice(grid, (B, H, N // 2, D)) * 2.0 ** -5
    k = np.concatenate([half, -half], axis=2)                     # channel means exactly zero
    v = rng.choice(grid, (B, H, N, D)) * 2.0 ** -3
    # the largest magnitude of every group is exactly 448 * 2^e for its exponent
    q[..., 0, 0] = 448.0 * 2.0 ** -4
    k[..., 0, 0], k[..., N // 2, 0] = 448.0 * 2.0 ** -5, -448.0 * 2.0 ** -5
    v[..., 0, :] = 448.0 * 2.0 ** -3
    quant = f8.quantize_qkv(q, k, v, S)
    assert np.array_equal(quant["q_hat"], q) and np.array_equal(quant["k_hat"], k)
    assert np.array_equal(quant["v_hat"], v)
    kept = [[[[0, 1, 3], [2], [1, 2, 3], [0]] for _ in range(H)]]
    got, _ = f8.fp8_block_sparse_attention(quant, kept, S, 0.35)
    want, _ = oracle.block_sparse_attention(q, k, v, kept, S, 0.35)
    assert np.array_equal(got, want)


def _f32(x):
    """float32 rounding by the C library's double -> float conversion."""
    return struct.unpack("<f", struct.pack("<f", float(x)))[0]


def test_softmax_scale_log2_closed_forms():
    """lambda = c * log2(e) in float32: 1/(sqrt(D) ln 2) for the default scale
    and c/ln 2 for a given one, within half a float32 ulp."""
    for D in (64, 112, 128):
        lam = f8.softmax_scale_log2(D)
        exact = 1.0 / (math.sqrt(D) * math.log(2.0))
        assert lam == _f32(lam) and abs(lam - exact) <= 2.0 ** -24 * exact, D
    lam = f8.softmax_scale_log2(128, 0.5)
    assert lam == _f32(lam) and abs(lam - 0.5 / math.log(2.0)) <= 2.0 ** -24 * lam
    assert f8.softmax_scale_log2(64) == _f32(0.125 / math.log(2.0))        # 1/8 is exact


def test_fold_scale_rounds_once_to_float32():
    """float32(q * lam) against the C library's conversion of the exact
    product, including a product exactly half-way between two float32 values
    (ties to even)."""
    rng = np.random.default_rng(8)
    q = _bf16(rng.standard_normal(500) * 4)
    for lam in (f8.softmax_scale_log2(128), f8.softmax_scale_log2(112), _f32(0.7213475)):
        got = f8.fold_scale(q, lam)
        for x, g in zip(q, got):
            assert g == _f32(float(x) * lam)
    # (1 + 2^-7)(1 + 2^-17) = 1 + 2^-7 + 2^-17 + 2^-24: half a float32 ulp above
    # a value with an even last bit
    tie = f8.fold_scale(np.array([1.0 + 2.0 ** -7]), 1.0 + 2.0 ** -17)[0]
    assert tie == 1.0 + 2.0 ** -7 + 2.0 ** -17
    # (1 + 2^-7)(1 + 2^-17 + 2^-23) = 1 + 2^-7 + 2^-17 + 2^-23 + 2^-24 + 2^-30:
    # more than half an ulp above 1 + 2^-7 + 2^-17 + 2^-23, so it rounds up
    up = f8.fold_scale(np.array([1.0 + 2.0 ** -7]), 1.0 + 2.0 ** -17 + 2.0 ** -23)[0]
    assert up == 1.0 + 2.0 ** -7 + 2.0 ** -17 + 2.0 ** -22


def test_quantize_q_with_folded_scale_pure_python():
    """Q's exponents and codes when it carries lambda, element by element in
    pure Python: the float32 product first, then the block grouping."""
    rng = np.random.default_rng(9)
    B, H, N, D, S = 1, 2, 10, 4, 4
    q = _bf16(rng.standard_normal((B, H, N, D)) * 3)
    k = _bf16(rng.standard_normal((B, H, N, D)))
    v = _bf16(rng.standard_normal((B, H, N, D)))
    lam = f8.softmax_scale_log2(D)
    out = f8.quantize_qkv(q, k, v, S, lam=lam)
    table = _finite_table()
    for h in range(H):
        qs = [[_f32(float(q[0, h, n, d]) * lam) for d in range(D)] for n in range(N)]
        for i, a in enumerate(range(0, N, S)):
            z = min(N, a + S)
            qa = max(abs(qs[n][d]) for n in range(a, z) for d in range(D))
            eq = next(e for e in range(-127, 128) if qa <= 448 * 2.0 ** e)
            assert out["q_exp"][0, h, i] == eq
            for n in range(a, z):
                for d in range(D):
                    assert out["q_code"][0, h, n, d] == _nearest_even(qs[n][d] * 2.0 ** -eq, table)


def test_folded_scale_attention_equals_plain_attention():
    """With lambda = 2^-3 and Q on the e4m3 grid, Q * lambda stays on it: the
    attention of the quantised inputs with logits ln2 * (q_hat . k_hat) equals
    plain attention with scale ln2 / 8."""
    rng = np.random.default_rng(10)
    B, H, N, D, S = 1, 2, 32, 8, 8
    grid = np.array([v for v in _finite_table().values() if abs(v) >= 2.0 ** -3])
    q = rng.choice(grid, (B, H, N, D)) * 2.0 ** -1
    half = rng.choice(grid, (B, H, N // 2, D)) * 2.0 ** -5
    k = np.concatenate([half, -half], axis=2)
    v = rng.choice(grid, (B, H, N, D)) * 2.0 ** -3
    q[..., 0, 0] = 448.0 * 2.0 ** -1
    k[..., 0, 0], k[..., N // 2, 0] = 448.0 * 2.0 ** -5, -448.0 * 2.0 ** -5
    v[..., 0, :] = 448.0 * 2.0 ** -3
    quant = f8.quantize_qkv(q, k, v, S, lam=0.125)
    assert np.array_equal(quant["q_hat"], q * 0.125)
    kept = [[[[0, 1, 3], [2], [1, 2, 3], [0]] for _ in range(H)]]
    got, gl = f8.fp8_block_sparse_attention(quant, kept, S, f8.LN2)
    want, wl = oracle.block_sparse_attention(q, k, v, kept, S, f8.LN2 / 8)
    assert np.array_equal(got, want) and np.array_equal(gl, wl)
