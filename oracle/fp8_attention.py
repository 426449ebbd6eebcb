"""8-bit (fp8 e4m3) block-sparse attention: quantisation and the attention it
feeds (oracle; test infrastructure only).

Section 4.2.4 (Quantization) points to the SageAttention series for attention:
8-bit (down to 4-bit) attention with outlier smoothing.  The paper gives no
formula; readings taken here (the design notes list them):

* format: e4m3 as the OCP 8-bit floating-point format defines it -- sign bit,
  4 exponent bits with bias 7, 3 mantissa bits; exponent field 0 encodes the
  subnormals m/8 * 2^-6; the all-ones pattern S.1111.111 is NaN; the largest
  finite magnitude is 1.75 * 2^8 = 448.  Values are rounded to the nearest
  e4m3 value, ties to the even code.
* scales are powers of two 2^e, e in [-127, 127]: for a group of values with
  largest magnitude a, e is the smallest exponent with a <= 448 * 2^e (e = 0
  for an all-zero group), and a value x is stored as the code of x * 2^-e.
* Q carries the softmax scale: it is multiplied by lambda = c * log2(e)
  (rounded once to float32) before it is quantised, so the matrix product of
  the codes is the logit in base-2 units and the probabilities are powers of
  two of it.  The product of a bf16 value and lambda is rounded once to
  float32, the quantiser's working precision.  Then one scale per (b, h,
  query block of S tokens), over the block's valid tokens and all channels.
* K, outlier smoothing: the per-(b, h) channel mean of K over all N tokens,
  rounded to bf16, is subtracted first (every logit of a query moves by the
  same amount, so the softmax is unchanged); the difference is taken in
  float32 (round to nearest even), the quantiser's working precision.  Then
  one scale per (b, h, key block).
* V: one scale per (b, h, channel) over all N tokens.
* attention: the block-sparse attention of the dequantised Q, K, V (the plain
  float64 definition of the sparse path), with logits ln(2) * (q_hat . k_hat)
  when Q carries lambda.  The GPU additionally rounds the
  unnormalised probabilities to e4m3 before the PV product; the tests bound
  that rounding's effect, the oracle keeps them exact.
"""
from __future__ import annotations

import math

import numpy as np

from .attention import block_sparse_attention
from .blocks import block_bounds
from .qknorm_rope import round_bf16

E4M3_MAX = 448.0
E_MIN, E_MAX = -127, 127
LOG2E = 1.4426950408889634          # log2(e), the float64 nearest to it
LN2 = math.log(2.0)


def softmax_scale_log2(head_dim: int, softmax_scale: float = 0.0) -> float:
    """lambda = c * log2(e) rounded once to float32, where c is the softmax
    scale: softmax_scale (a float32 value) when positive, else 1/sqrt(D),
    both in float64."""
    c = float(np.float32(softmax_scale)) if softmax_scale > 0 else 1.0 / math.sqrt(head_dim)
    return float(np.float32(c * LOG2E))


def fold_scale(q, lam: float) -> np.ndarray:
    """float32(q * lam) as float64, for bf16 values q and a float32 lam: the
    product of an 8-bit and a 24-bit significand is exact in float64, and it
    is rounded once to float32 (nearest, ties to even)."""
    return (np.asarray(q, dtype=np.float64) * float(lam)).astype(np.float32).astype(np.float64)


def e4m3_value(code: int) -> float:
    """The value of an e4m3 code (NaN for the two NaN patterns)."""
    code = int(code) & 0xFF
    sign = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return float("nan")
    if e == 0:
        return sign * (m / 8.0) * 2.0 ** -6
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


def round_e4m3(x: np.ndarray) -> np.ndarray:
    """Round float64 values with |x| <= 448 to the nearest e4m3 value (ties
    to even), as float64.  The spacing of e4m3 values near x is 2^(E-3) for
    |x| in [2^E, 2^(E+1)), E >= -6, and 2^-9 below 2^-6 (the subnormals)."""
    x = np.asarray(x, dtype=np.float64)
    if np.any(np.abs(x) > E4M3_MAX):
        raise ValueError("value outside the e4m3 range")
    out = np.zeros_like(x)
    nz = x != 0
    _, e = np.frexp(x[nz])                       # |x| = f * 2^e, f in [0.5, 1): E = e - 1
    q = np.ldexp(1.0, np.maximum(e - 4, -9))
    out[nz] = np.rint(x[nz] / q) * q             # np.rint: half to even
    return out


def encode_e4m3(x: np.ndarray) -> np.ndarray:
    """uint8 codes of values already on the e4m3 grid (|x| <= 448)."""
    x = np.asarray(x, dtype=np.float64)
    table = {}
    for c in range(256):
        v = e4m3_value(c)
        if v == v:                                # skip NaN
            table.setdefault(v, c)                # +0 -> 0x00 (first), -0 == +0
    out = np.empty(x.shape, dtype=np.uint8)
    flat = x.reshape(-1)
    o = out.reshape(-1)
    for n, v in enumerate(flat):
        c = table[float(v)]
        if v == 0 and np.signbit(v):
            c = 0x80
        o[n] = c
    return out


def scale_exponent(amax: float) -> int:
    """Smallest e in [-127, 127] with amax <= 448 * 2^e (0 for amax = 0).
    448 = 0.875 * 2^9 and amax = f * 2^ex with f in [0.5, 1), so the
    condition holds at e = ex - 9 when f <= 0.875 and at e = ex - 8 otherwise;
    both sides are exact."""
    amax = float(amax)
    if amax == 0.0:
        return 0
    f, ex = np.frexp(amax)
    e = int(ex) - 9 if f <= 0.875 else int(ex) - 8
    return max(E_MIN, min(E_MAX, e))


def quantize_groups(x: np.ndarray, exps: np.ndarray) -> np.ndarray:
    """Dequantised values 2^e * round_e4m3(x * 2^-e) (x, exps broadcastable)."""
    x = np.asarray(x, dtype=np.float64)
    s = np.ldexp(1.0, np.asarray(exps))
    return round_e4m3(x / s) * s


def k_smooth_mean(k: np.ndarray) -> np.ndarray:
    """K [B, H, N, D] -> per-(b, h) channel mean over N, rounded to bf16: [B, H, D]."""
    return round_bf16(np.mean(np.asarray(k, dtype=np.float64), axis=2))


def quantize_qkv(q, k, v, block: int, lam=None):
    """Quantise Q, K, V [B, H, N, D] (float64 holding bf16 values).  With lam
    (softmax_scale_log2), Q is first folded to float32(Q * lam): q_hat is
    then in base-2 logit units and the attention takes scale LN2.

    Returns a dict with
      q_exp [B, H, nB], k_exp [B, H, nB], v_exp [B, H, D]   (int)
      k_mean [B, H, D]                                        (bf16 values)
      q_hat, k_hat, v_hat [B, H, N, D]  dequantised values (2^e * code value)
      q_code, k_code, v_code [B, H, N, D]  code values (the e4m3 numbers)
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    if lam is not None:
        q = fold_scale(q, lam)
    B, H, N, D = q.shape
    bounds = block_bounds(N, block)
    nb = len(bounds)
    k_mean = k_smooth_mean(k)
    # the smoothing difference in float32 (both operands are bf16 values)
    ks = (k.astype(np.float32) - k_mean[:, :, None, :].astype(np.float32)).astype(np.float64)
    q_exp = np.zeros((B, H, nb), dtype=np.int64)
    k_exp = np.zeros((B, H, nb), dtype=np.int64)
    for b in range(B):
        for h in range(H):
            for i, (a, z) in enumerate(bounds):
                q_exp[b, h, i] = scale_exponent(np.abs(q[b, h, a:z]).max())
                k_exp[b, h, i] = scale_exponent(np.abs(ks[b, h, a:z]).max())
    v_exp = np.zeros((B, H, D), dtype=np.int64)
    for b in range(B):
        for h in range(H):
            for d in range(D):
                v_exp[b, h, d] = scale_exponent(np.abs(v[b, h, :, d]).max())
    tok_block = np.repeat(np.arange(nb), [z - a for a, z in bounds])
    qe = q_exp[:, :, tok_block][..., None]
    ke = k_exp[:, :, tok_block][..., None]
    ve = v_exp[:, :, None, :]
    q_code = round_e4m3(np.ldexp(q, -qe))
    k_code = round_e4m3(np.ldexp(ks, -ke))
    v_code = round_e4m3(np.ldexp(v, -ve))
    return {
        "q_exp": q_exp, "k_exp": k_exp, "v_exp": v_exp, "k_mean": k_mean,
        "q_code": q_code, "k_code": k_code, "v_code": v_code,
        "q_hat": np.ldexp(q_code, qe), "k_hat": np.ldexp(k_code, ke), "v_hat": np.ldexp(v_code, ve),
    }


def fp8_block_sparse_attention(quant: dict, kept, block: int, scale: float, rows=None):
    """Block-sparse attention of the dequantised tensors (float64); scale is
    LN2 when Q carries lambda."""
    return block_sparse_attention(quant["q_hat"], quant["k_hat"], quant["v_hat"], kept, block,
                                  scale, rows=rows)
