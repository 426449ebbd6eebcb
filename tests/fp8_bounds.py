"""What 8-bit quantisation itself does to attention (test infrastructure).

The fp8 path stores Q (times lambda = c log2 e, rounded to float32), K minus
its bf16 channel mean (rounded to float32) and V as e4m3 codes with one
power-of-two scale 2^E per group (Section 4.2.4; oracle/fp8_attention.py).
Rounding to the nearest e4m3 value errs by at most half a step: 2^-4 |x| in
the normal range (3 mantissa bits) and 2^-10 * 2^E among the subnormals
(spacing 2^-9 * 2^E), so for every stored value

    |x_hat - x| <= e(x) = max(2^-4 |x|, 2^(E - 10)),

plus 2^-24 |x| for the float32 product or difference taken first.  From that:

  logit of query n and key m, base 2 (the codes' product is the logit):
      |delta_nm| <= Delta_nm = sum_d e_q,nd |k_md| + |q_nd| e_k,md + e_q,nd e_k,md
                               + 2^-22 |q_n . k_m|     (lambda against c log2 e)
  weights: w_hat_m = w_m r_m with r_m in [exp(-L_m), exp(L_m)], L = ln2 Delta;
  with p the exact softmax and R in [R_lo, R_hi] = sum_m p_m exp(-/+ L_m),
      |p_hat_m - p_m| <= p_m max(exp(L_m)/R_lo - 1, 1 - exp(-L_m)/R_hi),
      p_hat_m <= p_m exp(L_m) / R_lo;
  output (sum_m (p_hat_m - p_m) = 0):
      |O_hat_e - O_e| <= sum_m |p_hat_m - p_m| |V_me - O_e| + sum_m p_hat_m e_v,me.

That is a worst case (every error aligned).  Taken as independent and
uniform in [-e, e] (variance e^2/3), the first-order spread of the same
errors is
      var(O_e) ~ sum_m p_m^2 ((ln2)^2 var(delta_nm) (V_me - O_e)^2 + var(v_me)),
      var(delta_nm) = sum_d (e_q,nd^2 k_md^2 + q_nd^2 e_k,md^2) / 3,
a model of the RMS error, not a bound; the errors being sums of many
independent bounded terms, no element should stray past SIGMAS standard
deviations of it, which the tests use as the per-element bound.
"""
from __future__ import annotations

import numpy as np

LN2 = float(np.log(2.0))
SIGMAS = 6.0          # per-element bound, in standard deviations of the error model


def element_error(x, exps) -> np.ndarray:
    """max(2^-4 |x|, 2^(E - 10)) for values x stored in groups of scale 2^E."""
    x = np.abs(np.asarray(x, dtype=np.float64))
    return np.maximum(2.0 ** -4 * x, np.ldexp(1.0, np.asarray(exps) - 10))


def storage_errors(q_fold, q_exp, k_smooth, k_exp, v, v_exp):
    """Per-value error bounds (e_q [n, D], e_k [m, D], e_v [m, D]) of the
    stored Q (float32(Q lambda), exponents q_exp [n]), K (float32(K - mean),
    exponents k_exp [m]) and V (channel exponents v_exp [D])."""
    q = np.asarray(q_fold, dtype=np.float64)
    k = np.asarray(k_smooth, dtype=np.float64)
    eq = element_error(q, np.asarray(q_exp)[:, None]) + 2.0 ** -24 * np.abs(q)
    ek = element_error(k, np.asarray(k_exp)[:, None]) + 2.0 ** -24 * np.abs(k)
    ev = element_error(v, np.asarray(v_exp)[None, :])
    return eq, ek, ev


def quantisation_effect(q_fold, eq, k_smooth, ek, v, ev, p, o):
    """Worst-case bound and first-order RMS model of |O_hat - O| for a set of
    queries against a set of keys.

    q_fold  : [n, D] float32(Q lambda) of the queries (base-2 logit units)
    k_smooth: [m, D] float32(K - mean) of the keys
    v       : [m, D] the keys' values
    eq, ek, ev : their storage error bounds (storage_errors)
    p       : [n, m] the exact softmax weights (rows summing to 1)
    o       : [n, D] the exact output
    returns (bound [n, D], variance [n, D])
    """
    q = np.asarray(q_fold, dtype=np.float64)
    k = np.asarray(k_smooth, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    aq, ak = np.abs(q), np.abs(k)
    delta = eq @ ak.T + aq @ ek.T + eq @ ek.T + 2.0 ** -22 * np.abs(q @ k.T)      # [n, m]
    lam_n = LN2 * delta
    r_lo = (p * np.exp(-lam_n)).sum(axis=1, keepdims=True)
    r_hi = (p * np.exp(lam_n)).sum(axis=1, keepdims=True)
    dp = p * np.maximum(np.exp(lam_n) / r_lo - 1.0, 1.0 - np.exp(-lam_n) / r_hi)
    p_hi = p * np.exp(lam_n) / r_lo
    dev = np.abs(v[None, :, :] - o[:, None, :])                                   # [n, m, D]
    bound = np.einsum("nm,nmd->nd", dp, dev) + p_hi @ ev
    var_delta = ((eq * eq) @ (k * k).T + (q * q) @ (ek * ek).T) / 3.0             # [n, m]
    var = (LN2 ** 2) * np.einsum("nm,nmd->nd", p * p * var_delta, dev * dev) + (p * p) @ (ev * ev / 3.0)
    return bound, var


def exact_attention(q, k, v, scale):
    """Softmax attention in float64: (weights [n, m], output [n, D], lse [n])."""
    s = scale * (np.asarray(q, dtype=np.float64) @ np.asarray(k, dtype=np.float64).T)
    mx = s.max(axis=1, keepdims=True)
    w = np.exp(s - mx)
    l = w.sum(axis=1, keepdims=True)
    return w / l, (w @ np.asarray(v, dtype=np.float64)) / l, mx[:, 0] + np.log(l[:, 0])
