"""Pins of the fp8 quantisation bounds in tests/fp8_bounds.py (what e4m3
storage of Q, K and V does to attention, derived from the format's step).

  - the per-value bound max(2^-4 |x|, 2^(E-10)) holds for every rounding the
    oracle's quantiser makes and is reached (half a step at the midpoints);
  - on seeded cases (plain, a key sink scaled by 3, values deep in the
    subnormal range, large logits) the dequantised attention stays within
    the worst-case bound of the exact attention in every element (all errors
    aligned: rigorous, and 30-100 times the observed error);
  - the first-order model of the error's spread predicts the observed RMS
    within a factor of two either way (measured 0.66-0.74), and no element
    exceeds six of its standard deviations (measured at most 3.5): the
    six-sigma form is the per-element bound the GPU tests use;
  - a planted mistake in the model (V's storage error left out) breaks the
    six-sigma bound.
"""
import math

import numpy as np
import pytest

import oracle.fp8_attention as of8

from . import fp8_bounds as fb

pytestmark = pytest.mark.cpu


def test_element_error_bounds_every_rounding():
    rng = np.random.default_rng(5)
    worst = 0.0
    for e in (-20, -7, -3, 0, 2, 9):
        x = np.concatenate([rng.uniform(-448, 448, 20000), rng.uniform(-2.0 ** -6, 2.0 ** -6, 20000),
                            (np.arange(-4096, 4096) + 0.5) * 2.0 ** -9])       # subnormal midpoints
        xs = np.ldexp(x, e)
        got = of8.quantize_groups(xs, e)
        err = np.abs(got - xs)
        b = fb.element_error(xs, e)
        assert np.all(err <= b), e
        worst = max(worst, float(np.max(err / b)))
    assert worst > 0.99


def _case(kind, seed=7, N=256, D=32, S=64):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((N, D))
    k = rng.standard_normal((N, D))
    v = rng.standard_normal((N, D))
    if kind == "sink":
        k[:32] *= 3.0
    elif kind == "tiny":
        v *= 1e-3
        v[:, :4] *= 1e-4                       # channels far below their group's largest value
        k[:, :8] *= 1e-3
    elif kind == "large_logits":
        q *= 3.0
        k *= 3.0
    # the values are bf16 numbers, as the path's inputs are
    r = lambda a: (a.astype(np.float32).view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32).astype(np.float64)
    return r(q), r(k), r(v), S


def _effect(q, k, v, S, drop=None):
    """(|O_hat - O|, bound, variance) of one head; drop names a storage error
    to leave out of the bound (a planted mistake)."""
    N, D = q.shape
    c = 1.0 / math.sqrt(D)
    lam = of8.softmax_scale_log2(D)
    quant = of8.quantize_qkv(q[None, None], k[None, None], v[None, None], S, lam=lam)
    qf = of8.fold_scale(q, lam)
    ks = (k.astype(np.float32) - quant["k_mean"][0, 0].astype(np.float32)).astype(np.float64)
    tok_block = np.arange(N) // S
    p, o, _ = fb.exact_attention(q, k, v, c)
    _, o_hat, _ = fb.exact_attention(quant["q_hat"][0, 0], quant["k_hat"][0, 0], quant["v_hat"][0, 0], of8.LN2)
    eq, ek, ev = fb.storage_errors(qf, quant["q_exp"][0, 0][tok_block], ks, quant["k_exp"][0, 0][tok_block],
                                   v, quant["v_exp"][0, 0])
    if drop == "v":
        ev = np.zeros_like(ev)
    elif drop == "k":
        ek = np.zeros_like(ek)
    bound, var = fb.quantisation_effect(qf, eq, ks, ek, v, ev, p, o)
    return np.abs(o_hat - o), bound, var


@pytest.mark.parametrize("kind", ["plain", "sink", "tiny", "large_logits"])
def test_dequantised_attention_within_the_bounds(kind):
    err, bound, var = _effect(*_case(kind))
    assert np.all(err <= bound), (kind, float((err - bound).max()))
    assert np.all(err <= fb.SIGMAS * np.sqrt(var)), (kind, float((err / np.sqrt(var)).max()))
    rms, model = float(np.sqrt(np.mean(err ** 2))), float(np.sqrt(np.mean(var)))
    assert 0.5 * model < rms < 2.0 * model, (kind, rms, model)


@pytest.mark.parametrize("kind", ["sink", "large_logits"])
def test_model_without_the_value_error_is_caught(kind):
    err, _, var = _effect(*_case(kind), drop="v")
    assert np.any(err > fb.SIGMAS * np.sqrt(var)), kind
