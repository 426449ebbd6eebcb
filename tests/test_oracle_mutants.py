"""Planted mistakes in the oracle must be caught by its pins.

Each case swaps one oracle function for a plausibly wrong version (dropped term,
wrong divisor, transposed operand, reversed tie-break, ...) on the CPU and runs
the pins that should fail.  A pin set that let a mutant through would not pin
the oracle.
"""
import math

import numpy as np
import pytest

import oracle
import oracle.attention as oatt
import oracle.blocks as oblk
import oracle.select as osel
import oracle.fp8_attention as of8

from . import test_oracle_attention as TA
from . import test_oracle_pool as TP
from . import test_oracle_select as TS
from . import test_oracle_fp8 as TF8

pytestmark = pytest.mark.cpu


def _pool_div_by_block(x, block):
    x = np.asarray(x, dtype=np.float64)
    b = oblk.block_bounds(x.shape[-2], block)
    out = np.empty(x.shape[:-2] + (len(b), x.shape[-1]))
    for i, (a, e) in enumerate(b):
        out[..., i, :] = x[..., a:e, :].sum(axis=-2) / block
    return out


def _scores_transposed(q, k, scale):
    return scale * np.matmul(np.asarray(k, float), np.swapaxes(np.asarray(q, float), -1, -2))


def _order_desc_high_index_wins(row, candidates):
    cand = np.asarray(list(candidates), dtype=np.int64)
    order = np.lexsort((-cand, -row[cand]))
    return [int(j) for j in cand[order]]


def _cummass_forced_mass_ignored(scores, tau, cap, forced=()):
    scores = np.asarray(scores, float)
    flat = scores.reshape(-1, scores.shape[-1])
    forced = sorted(set(forced))
    rows = []
    for s in flat:
        p = np.exp(s - s.max()); p /= p.sum()
        kept, mass = list(forced), 0.0
        for j in osel._order_desc(s, [j for j in range(len(s)) if j not in forced]):
            if mass >= tau or len(kept) >= cap:
                break
            kept.append(j); mass += p[j]
        rows.append(sorted(kept))
    return osel._reshape_nested(rows, scores.shape[:-1])


def _attend_no_max_in_lse(qrows, keys, vals, scale):
    logits = scale * (qrows @ keys.T)
    mx = logits.max(axis=1, keepdims=True)
    w = np.exp(logits - mx)
    return (w @ vals) / w.sum(1, keepdims=True), np.log(w.sum(1))


def _attend_scale_dropped(qrows, keys, vals, scale):
    logits = qrows @ keys.T
    mx = logits.max(axis=1, keepdims=True)
    w = np.exp(logits - mx)
    return (w @ vals) / w.sum(1, keepdims=True), mx[:, 0] + np.log(w.sum(1))


def _attend_values_unnormalised(qrows, keys, vals, scale):
    logits = scale * (qrows @ keys.T)
    mx = logits.max(axis=1, keepdims=True)
    w = np.exp(logits - mx)
    return w @ vals, mx[:, 0] + np.log(w.sum(1))


def _bounds_off_by_one(seq_len, block):
    nb = -(-seq_len // block)
    return [(i * block, min((i + 1) * block, seq_len - 1)) for i in range(nb)]


MUTANTS = [
    ("pool divides by S", oblk, "pool_blocks", _pool_div_by_block,
     [lambda g: TP.test_pool_arithmetic_progression_closed_form(),
      lambda g: TS.test_golden_pool_then_topk(g)]),
    ("scores transposed", osel, "block_scores", _scores_transposed,
     [lambda g: TS.test_scores_bruteforce_and_orientation(), lambda g: TS.test_golden_pool_then_topk(g)]),
    ("ties go to the higher index", osel, "_order_desc", _order_desc_high_index_wins,
     [lambda g: TS.test_topk_bruteforce_random_and_ties(), lambda g: TS.test_golden_pool_then_topk(g),
      lambda g: TS.test_golden_mass(g)]),
    ("forced mass not counted", osel, "select_cummass", _cummass_forced_mass_ignored,
     [lambda g: TS.test_golden_mass(g),
      lambda g: TS.test_mass_matches_independent_search_and_invariants(0.9, 0.3, True)]),
    ("LSE without the max", oatt, "_attend", _attend_no_max_in_lse,
     [lambda g: TA.test_sparse_bruteforce_pure_python(), lambda g: TA.test_dense_matches_torch_sdpa_float64()]),
    ("softmax scale dropped", oatt, "_attend", _attend_scale_dropped,
     [lambda g: TA.test_sparse_bruteforce_pure_python(), lambda g: TA.test_scale_is_applied()]),
    ("values not normalised", oatt, "_attend", _attend_values_unnormalised,
     [lambda g: TA.test_constant_values_give_constant_output()]),
    ("last token of the sequence dropped", oblk, "block_bounds", _bounds_off_by_one,
     [lambda g: TP.test_num_blocks_closed_form(1000, 64)]),
]


@pytest.mark.parametrize("name,mod,attr,fn,pins", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(name, mod, attr, fn, pins, monkeypatch, golden_dir):
    monkeypatch.setattr(mod, attr, fn)
    # re-export through the package namespace the pins call
    if hasattr(oracle, attr):
        monkeypatch.setattr(oracle, attr, fn)
    for mname in ("oracle.attention", "oracle.select", "oracle.blocks"):
        m = __import__(mname, fromlist=["x"])
        if hasattr(m, attr) and m is not mod:
            monkeypatch.setattr(m, attr, fn)
    for pin in pins:
        with pytest.raises(AssertionError):
            pin(golden_dir)


# ---- QKNorm + RoPE + pool ----
import oracle.qknorm_rope as oqr  # noqa: E402

from . import test_oracle_qknorm_rope as TQ  # noqa: E402


def _rope_half_split(x, angles):
    x = np.asarray(x, dtype=np.float64)
    h = x.shape[-1] // 2
    a, b = x[..., :h], x[..., h:]
    c, s = np.cos(angles), np.sin(angles)
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


_ORIG_APPLY_ROPE = oqr.apply_rope


def _rope_turned_backwards(x, angles):
    return _ORIG_APPLY_ROPE(x, -np.asarray(angles))
_ORIG_ROPE_ANGLES = oqr.rope_angles
_ORIG_RMS_NORM = oqr.rms_norm
_ORIG_ROUND = oqr.round_bf16


def _angles_axes_reversed(grid, head_dim, base):
    T, H, W = grid
    ang = _ORIG_ROPE_ANGLES((W, H, T), head_dim, base)      # x treated as t and t as x
    return ang.reshape(W, H, T, -1).transpose(2, 1, 0, 3).reshape(T * H * W, -1)


def _rms_norm_without_eps(x, gamma, eps):
    return _ORIG_RMS_NORM(x, gamma, 0.0)


def _rms_norm_without_gamma(x, gamma, eps):
    return _ORIG_RMS_NORM(x, np.ones_like(np.asarray(gamma, dtype=np.float64)), eps)


def _round_via_float32(x):
    return _ORIG_ROUND(np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64))


def _producer_pools_before_rounding(q, k, gamma_q, gamma_k, grid, block, eps, base):
    qx = oqr.norm_rope(q, gamma_q, grid, eps, base)
    kx = oqr.norm_rope(k, gamma_k, grid, eps, base)
    return (oqr.round_bf16(qx), oqr.round_bf16(kx), oqr.pool_blocks(qx, block), oqr.pool_blocks(kx, block))


QKR_MUTANTS = [
    ("RoPE pairs split in halves", "apply_rope", _rope_half_split,
     [TQ.test_rope_is_complex_multiplication]),
    ("RoPE turned backwards", "apply_rope", _rope_turned_backwards,
     [TQ.test_rope_is_complex_multiplication]),
    ("RoPE axes in x, y, t order", "rope_angles", _angles_axes_reversed,
     [TQ.test_rope_angles_hand_derived]),
    ("RMSNorm without eps", "rms_norm", _rms_norm_without_eps, [TQ.test_rms_norm_closed_forms]),
    ("RMSNorm without gamma", "rms_norm", _rms_norm_without_gamma, [TQ.test_rms_norm_closed_forms]),
    ("bf16 rounding through float32", "round_bf16", _round_via_float32,
     [TQ.test_round_bf16_ties_and_no_double_rounding]),
    ("pooled before rounding", "qknorm_rope_pool", _producer_pools_before_rounding,
     [TQ.test_producer_pools_its_rounded_outputs]),
]


@pytest.mark.parametrize("name,attr,fn,pins", QKR_MUTANTS, ids=[m[0] for m in QKR_MUTANTS])
def test_qknorm_rope_mutant_is_caught(name, attr, fn, pins, monkeypatch):
    monkeypatch.setattr(oqr, attr, fn)
    for pin in pins:
        with pytest.raises(AssertionError):
            pin()


# ---- token pruning ----
import oracle.token_prune as otp  # noqa: E402

from . import test_oracle_token_prune as TT  # noqa: E402

_ORIG_SELECT_TOKENS = otp.select_tokens


def _scores_over_tokens(x):
    x = np.asarray(x, dtype=np.float64)
    s = np.sum(x * x, axis=-2, keepdims=True)            # reduced over the wrong axis
    return np.broadcast_to(s[..., 0], x.shape[:-1]).copy()


def _select_high_index_wins(scores, k):
    scores = np.asarray(scores, dtype=np.float64)
    B, N = scores.shape
    out = np.empty((B, k), dtype=np.int64)
    idx = np.arange(N)
    for b in range(B):
        out[b] = np.sort(np.lexsort((-idx, -scores[b]))[:k])
    return out


def _select_unsorted(scores, k):
    scores = np.asarray(scores, dtype=np.float64)
    return np.stack([np.lexsort((np.arange(scores.shape[1]), -row))[:k] for row in scores])


def _keep_count_floor(n_tokens, keep_ratio):
    return max(1, min(int(n_tokens), int(math.floor(keep_ratio * n_tokens))))


def _scatter_without_base(y_kept, kept, base):
    out = np.zeros_like(np.asarray(base))
    for b in range(out.shape[0]):
        out[b, kept[b]] = y_kept[b]
    return out


TP_MUTANTS = [
    ("scores over the token axis", "token_scores", _scores_over_tokens,
     [TT.test_scores_are_squared_library_norms_and_closed_form]),
    ("token ties go to the higher index", "select_tokens", _select_high_index_wins,
     [TT.test_select_matches_python_sort_with_ties, TT.test_select_hand_worked]),
    ("kept tokens not in ascending order", "select_tokens", _select_unsorted,
     [TT.test_select_matches_python_sort_with_ties, TT.test_select_hand_worked]),
    ("keep count rounded down", "keep_count", _keep_count_floor, [TT.test_keep_count]),
    ("scatter drops the base rows", "scatter_tokens", _scatter_without_base,
     [TT.test_gather_scatter_identities]),
]


@pytest.mark.parametrize("name,attr,fn,pins", TP_MUTANTS, ids=[m[0] for m in TP_MUTANTS])
def test_token_prune_mutant_is_caught(name, attr, fn, pins, monkeypatch):
    monkeypatch.setattr(otp, attr, fn)
    for pin in pins:
        with pytest.raises(AssertionError):
            pin()


# ---- fp8 quantisation ----

def _e4m3_half_away(x):
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros_like(x)
    nz = x != 0
    _, e = np.frexp(x[nz])
    q = np.ldexp(1.0, np.maximum(e - 4, -9))
    out[nz] = np.sign(x[nz]) * np.floor(np.abs(x[nz]) / q + 0.5) * q
    return out


def _e4m3_subnormal_step_too_fine(x):
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros_like(x)
    nz = x != 0
    _, e = np.frexp(x[nz])
    q = np.ldexp(1.0, np.maximum(e - 4, -10))
    out[nz] = np.rint(x[nz] / q) * q
    return out


_true_scale_exponent = of8.scale_exponent


def _scale_exponent_floor(amax):
    if amax == 0:
        return 0
    return int(math.floor(math.log2(amax / 448.0)))


def _no_smoothing(k):
    k = np.asarray(k, dtype=np.float64)
    return np.zeros(k.shape[:2] + k.shape[3:])


def _fold_ignores_scale(q, lam):
    return np.asarray(q, dtype=np.float64)


def _fold_in_float64(q, lam):
    return np.asarray(q, dtype=np.float64) * float(lam)


FP8_MUTANTS = [
    ("softmax scale not folded into Q", "fold_scale", _fold_ignores_scale,
     [TF8.test_fold_scale_rounds_once_to_float32, TF8.test_quantize_q_with_folded_scale_pure_python,
      TF8.test_folded_scale_attention_equals_plain_attention]),
    ("folded Q not rounded to float32", "fold_scale", _fold_in_float64,
     [TF8.test_fold_scale_rounds_once_to_float32]),
    ("e4m3 ties away from zero", "round_e4m3", _e4m3_half_away,
     [TF8.test_rounding_matches_brute_force_nearest_even]),
    ("e4m3 subnormal spacing 2^-10", "round_e4m3", _e4m3_subnormal_step_too_fine,
     [TF8.test_rounding_matches_brute_force_nearest_even]),
    ("scale exponent rounded down", "scale_exponent", _scale_exponent_floor,
     [TF8.test_scale_exponent_brute_force]),
    ("no K smoothing", "k_smooth_mean", _no_smoothing,
     [TF8.test_quantize_qkv_matches_pure_python_grouping]),
]


@pytest.mark.parametrize("name,attr,fn,pins", FP8_MUTANTS, ids=[m[0] for m in FP8_MUTANTS])
def test_fp8_mutant_is_caught(name, attr, fn, pins, monkeypatch):
    monkeypatch.setattr(of8, attr, fn)
    for pin in pins:
        with pytest.raises((AssertionError, ValueError)):
            pin()


# ---- first-order remainder of dropped blocks ----
import oracle.remainder as orem  # noqa: E402

from . import test_oracle_remainder as TR  # noqa: E402


def _moment_times_query_transposed(mom, qr):
    return np.einsum("jde,nd->nje", mom, qr)


def _no_first_order(mom, qr):
    return np.zeros((qr.shape[0], mom.shape[0], mom.shape[1]))


def _moment_sign_flipped(mom, qr):
    return -np.einsum("jed,nd->nje", mom, qr)


def _block_counts_ignored(count):
    return np.zeros_like(count)


def _moments_not_centred(k, v, block):
    kbar, vbar, _ = _ORIG_BLOCK_MOMENTS(k, v, block)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    b = oblk.block_bounds(k.shape[-2], block)
    m = np.stack([np.matmul(np.swapaxes(v[..., a:e, :], -1, -2), k[..., a:e, :]) for a, e in b], axis=-3)
    return kbar, vbar, m


_ORIG_BLOCK_MOMENTS = orem.block_moments

def _weight_at_block_mean(qr, qbar_i, kbar_drop, scale, weight):
    return _ORIG_FIRST_ORDER_LOG_WEIGHTS(qr, qbar_i, kbar_drop, scale, "block_mean")


def _weight_at_query_always(qr, qbar_i, kbar_drop, scale, weight):
    return _ORIG_FIRST_ORDER_LOG_WEIGHTS(qr, qbar_i, kbar_drop, scale, "query")


_ORIG_FIRST_ORDER_LOG_WEIGHTS = orem.first_order_log_weights

REM_MUTANTS = [
    ("moment applied transposed", "moment_times_query", _moment_times_query_transposed,
     [lambda: TR.test_error_is_second_order(True, "query"), lambda: TR.test_error_is_second_order(False, "query"),
      lambda: TR.test_first_order_term_by_term()]),
    ("first-order term dropped", "moment_times_query", _no_first_order,
     [lambda: TR.test_error_is_second_order(True, "query"), lambda: TR.test_error_is_second_order(False, "query"),
      lambda: TR.test_error_is_second_order(True, "block_mean"), lambda: TR.test_first_order_term_by_term()]),
    ("first-order term with the wrong sign", "moment_times_query", _moment_sign_flipped,
     [lambda: TR.test_error_is_second_order(True, "query"), lambda: TR.test_first_order_term_by_term()]),
    ("dropped block counted as one token", "log_token_count", _block_counts_ignored,
     [lambda: TR.test_constant_key_blocks_equal_dense(37, 8, "query"),
      lambda: TR.test_constant_key_blocks_equal_dense(9, 4, "block_mean"), lambda: TR.test_first_order_term_by_term()]),
    ("moments about zero, not the block mean", "block_moments", _moments_not_centred,
     [lambda: TR.test_moments_bruteforce_and_identity(), lambda: TR.test_constant_key_blocks_equal_dense(40, 8, "query")]),
    ("first-order weight at the block-mean query", "first_order_log_weights", _weight_at_block_mean,
     [lambda: TR.test_plain_expansion_is_second_order_in_the_key_deviation(),
      lambda: TR.test_first_order_term_by_term()]),
    ("block-mean form computed with the query's own weight", "first_order_log_weights", _weight_at_query_always,
     [lambda: TR.test_block_mean_form_is_first_order_in_the_key_deviation()]),
]


@pytest.mark.parametrize("name,attr,fn,pins", REM_MUTANTS, ids=[m[0] for m in REM_MUTANTS])
def test_remainder_mutant_is_caught(name, attr, fn, pins, monkeypatch):
    monkeypatch.setattr(orem, attr, fn)
    for pin in pins:
        with pytest.raises(AssertionError):
            pin()
