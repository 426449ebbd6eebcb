"""QK RMSNorm + 3-D rotary position embedding + block pooling (oracle; test
infrastructure only).

The paper names this fusion but prints no formula for it: Section 4.2.5
(Kernel Fusion) gives "fused RoPE + norm" as a typical fusion candidate, and
Appendix A.2.2 lists fused QKNorm+RoPE among the lossless kernels of the
LTX-2.3 stack.  Fusing the block pooling of Section 4.2.2 into the same pass
means Q and K are read once for both.  Readings taken here (the design notes
list them):

* RMSNorm per token over the head dimension:
      y = x / sqrt(mean_d(x_d^2) + eps) * gamma,   gamma [D] shared by heads.
* 3-D RoPE on interleaved pairs (x[2p], x[2p+1]), p = 0 .. D/2-1.  The pairs
  are cut into three contiguous groups for the t, y and x axes, of sizes
      n_t = D/2 - 2*floor(D/6),  n_y = n_x = floor(D/6),
  and pair i of a group of size n turns by the angle pos * base^(-i/n), pos
  being the token's integer coordinate on that axis (t-major raster order:
  n = (t*H + y)*W + x).  A turn by phi maps (a, b) to
  (a cos phi - b sin phi, a sin phi + b cos phi).
* The result is rounded once to bf16 (round to nearest, ties to even).
* The block summaries are the means (over valid tokens) of those rounded
  outputs, i.e. block pooling applied to what is written.
"""
from __future__ import annotations


import numpy as np

from .blocks import pool_blocks


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (ties to even), returned
    as float64.  bf16 keeps 8 significant bits and float32's exponent range;
    this rounds from float64 directly (no intermediate float32 rounding)."""
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros_like(x)
    nz = x != 0
    m, e = np.frexp(x[nz])                      # x = m * 2^e, 0.5 <= |m| < 1
    # spacing of bf16 values around x: 2^(e-8) for normal numbers, never below
    # the subnormal spacing 2^-133
    q = np.ldexp(1.0, np.maximum(e - 8, -133))
    out[nz] = np.rint(x[nz] / q) * q            # np.rint rounds half to even
    return out


def rms_norm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """x [..., D] -> x / sqrt(mean(x^2) + eps) * gamma, in float64."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gamma, dtype=np.float64)


def rope_pair_groups(head_dim: int):
    """(n_t, n_y, n_x): how many rotation pairs each axis gets."""
    half = head_dim // 2
    n_yx = head_dim // 6
    return half - 2 * n_yx, n_yx, n_yx


def rope_angles(grid, head_dim: int, base: float) -> np.ndarray:
    """Rotation angle of every (token, pair): float64 [T*H*W, D/2]."""
    T, H, W = grid
    n_t, n_y, n_x = rope_pair_groups(head_dim)
    t, y, x = np.meshgrid(np.arange(T), np.arange(H), np.arange(W), indexing="ij")
    pos = [t.reshape(-1).astype(np.float64), y.reshape(-1).astype(np.float64),
           x.reshape(-1).astype(np.float64)]
    cols = []
    for axis, n in enumerate((n_t, n_y, n_x)):
        inv = np.power(float(base), -np.arange(n, dtype=np.float64) / n)
        cols.append(pos[axis][:, None] * inv[None, :])
    return np.concatenate(cols, axis=1)


def apply_rope(x: np.ndarray, angles: np.ndarray) -> np.ndarray:
    """Turn each interleaved pair of x [..., N, D] by angles [N, D/2]."""
    x = np.asarray(x, dtype=np.float64)
    a, b = x[..., 0::2], x[..., 1::2]
    c, s = np.cos(angles), np.sin(angles)
    out = np.empty_like(x)
    out[..., 0::2] = a * c - b * s
    out[..., 1::2] = a * s + b * c
    return out


def norm_rope(x: np.ndarray, gamma: np.ndarray, grid, eps: float, base: float) -> np.ndarray:
    """RMSNorm then RoPE of x [B, H, N, D] (float64, not rounded)."""
    D = x.shape[-1]
    return apply_rope(rms_norm(x, gamma, eps), rope_angles(grid, D, base))


def qknorm_rope_pool(q, k, gamma_q, gamma_k, grid, block: int, eps: float, base: float):
    """The fused producer: (q_out, k_out, q_pool, k_pool), outputs as float64
    holding bf16 values, summaries as float64 means of those outputs."""
    q_out = round_bf16(norm_rope(q, gamma_q, grid, eps, base))
    k_out = round_bf16(norm_rope(k, gamma_k, grid, eps, base))
    return q_out, k_out, pool_blocks(q_out, block), pool_blocks(k_out, block)
