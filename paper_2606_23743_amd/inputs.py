"""Seeded synthetic Q/K/V for video self-attention (the only module both the
kernels' tests and the oracle are fed from; it holds none of the method's
arithmetic).

Recipe (per workload seed s):
  root = SeedSequence(s); smooth_seq, noise_seq = root.spawn(2)
  per head h (generator from smooth_seq.spawn(H)[h]):
      f   ~ U[0, 2)^(8 x 3)   cycles per axis (t, y, x) for 8 sinusoids
      phi ~ U[0, 2*pi)^8
      A   ~ N(0, 0.5^2)^(8 x D)  shared Q/K amplitudes
      A'  ~ N(0, 0.5^2)^(8 x D)  V amplitudes
      F[n, j] = sin(2*pi*(f_jt*t/T + f_jy*y/H + f_jx*x/W) + phi_j)   (n = (t*H + y)*W + x)
      smooth_qk = F @ A ; smooth_v = F @ A'         (unit RMS per channel)
  per (tensor, b, h) noise Z ~ N(0, 1) from noise_seq.spawn(3*B*H)[(tensor*B + b)*H + h]
      Q = 0.5*Z_q + smooth_qk ; K = 0.5*Z_k + smooth_qk ; V = 0.5*Z_v + smooth_v
  optional attention sink: K[:, :, :sink_tokens, :] *= sink_scale
  every tensor is rounded once, fp32 -> bf16 round-to-nearest-even.

Q and K share the smooth part, so attention concentrates on nearby tokens in
(t, y, x) the way a video DiT's does; every batch entry of a head reuses that
head's smooth part with fresh noise (the conditional/unconditional pair of a
classifier-free-guidance batch).

Outputs are bf16 bit patterns as uint16 numpy arrays [B, H, N, D]; `to_device`
wraps them as torch bfloat16 tensors.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict

import numpy as np

from .workloads import Workload

N_SINUSOIDS = 8
NOISE_STD = 0.5
AMP_STD = 0.5


def _round_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits, round to nearest even (inputs are finite)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def _grid_coords(t: int, h: int, w: int):
    tt, yy, xx = np.meshgrid(np.arange(t), np.arange(h), np.arange(w), indexing="ij")
    return (tt.reshape(-1) / t, yy.reshape(-1) / h, xx.reshape(-1) / w)


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def generate(wl: Workload, seed: int | None = None) -> Dict[str, np.ndarray]:
    """Return {"q","k","v"}: uint16 bf16 bits, shape [B, H, N, D], C-contiguous."""
    seed = wl.seed if seed is None else seed
    B, H, D = wl.batch, wl.heads, wl.head_dim
    N = wl.seq_len
    root = np.random.SeedSequence(seed)
    smooth_seq, noise_seq = root.spawn(2)
    head_seqs = smooth_seq.spawn(H)
    noise_seqs = noise_seq.spawn(3 * B * H)
    ct, cy, cx = _grid_coords(wl.grid_t, wl.grid_h, wl.grid_w)

    smooth_qk = []
    smooth_v = []
    for h in range(H):
        g = np.random.Generator(np.random.PCG64(head_seqs[h]))
        f = g.uniform(0.0, 2.0, size=(N_SINUSOIDS, 3))
        phi = g.uniform(0.0, 2.0 * np.pi, size=N_SINUSOIDS)
        a = g.normal(0.0, AMP_STD, size=(N_SINUSOIDS, D))
        a2 = g.normal(0.0, AMP_STD, size=(N_SINUSOIDS, D))
        arg = np.outer(ct, f[:, 0]) + np.outer(cy, f[:, 1]) + np.outer(cx, f[:, 2])
        F = np.sin(2.0 * np.pi * arg + phi[None, :])
        smooth_qk.append((F @ a).astype(np.float32))
        smooth_v.append((F @ a2).astype(np.float32))

    out = {name: np.empty((B, H, N, D), dtype=np.uint16) for name in ("q", "k", "v")}
    names = ("q", "k", "v")

    def fill(task):
        ti, b, h = task
        g = np.random.Generator(np.random.PCG64(noise_seqs[(ti * B + b) * H + h]))
        z = g.standard_normal((N, D), dtype=np.float32)
        z *= np.float32(NOISE_STD)
        z += smooth_v[h] if ti == 2 else smooth_qk[h]
        if ti == 1 and wl.sink_tokens > 0:
            z[: wl.sink_tokens] *= np.float32(wl.sink_scale)
        out[names[ti]][b, h] = _round_bf16(z)

    tasks = [(ti, b, h) for ti in range(3) for b in range(B) for h in range(H)]
    with ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(fill, tasks))
    return out


def hidden_states(batch: int, n_tokens: int, channels: int, seed: int,
                  dup_frac: float = 0.05, n_zero: int = 2) -> np.ndarray:
    """Seeded transformer hidden states, uint16 bf16 bits [B, N, C].

    Recipe: per token a log-normal scale exp(0.5 g), g ~ N(0, 1), times
    N(0, 1) channel values, rounded once to bf16; then per batch entry a
    fraction dup_frac of the tokens are overwritten with copies of other
    tokens' rows (bit-identical rows: exact score ties between tokens far
    apart), and n_zero tokens are set to zero rows (ties at the lowest score).
    """
    root = np.random.SeedSequence(seed)
    seqs = root.spawn(batch)
    out = np.empty((batch, n_tokens, channels), dtype=np.uint16)

    def fill(b):
        g = np.random.Generator(np.random.PCG64(seqs[b]))
        scale = np.exp(0.5 * g.standard_normal(n_tokens)).astype(np.float32)
        n_dup = int(dup_frac * n_tokens)
        dst = g.choice(n_tokens, size=n_dup + min(n_zero, n_tokens), replace=False)
        src = g.integers(0, n_tokens, size=n_dup)
        step = 8192
        for s0 in range(0, n_tokens, step):
            z = g.standard_normal((min(step, n_tokens - s0), channels), dtype=np.float32)
            z *= scale[s0:s0 + step, None]
            out[b, s0:s0 + step] = _round_bf16(z)
        out[b, dst[:n_dup]] = out[b, src]
        out[b, dst[n_dup:]] = 0

    with ThreadPoolExecutor(min(_workers(), batch)) as ex:
        list(ex.map(fill, range(batch)))
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32 (for plumbing and tests)."""
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_device(bits: np.ndarray, device="cuda"):
    """uint16 bf16 bits -> torch.bfloat16 tensor on `device` (same bytes)."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(bits)).view(torch.bfloat16)
    return t.to(device)
