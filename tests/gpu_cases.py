"""Shared plumbing for the GPU parity tests: build inputs, run the HIP path
through the C ABI, run the oracle on the same bytes.  The oracle and the HIP
path see identical bf16 inputs; nothing the GPU produces is fed to the oracle.
"""
from __future__ import annotations

import math
import sys

import numpy as np

import oracle
from paper_2606_23743_amd import inputs, workloads
import paper_2606_23743_amd as sva


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def device_inputs(bits):
    return {n: inputs.to_device(bits[n]) for n in ("q", "k", "v")}


def oracle_inputs_head(bits, b, h):
    return {n: oracle.bf16_bits_to_f64(bits[n][b, h]) for n in ("q", "k", "v")}


def oracle_pool_all(bits, block):
    """Oracle pooled Q and K for every (b, h): float64 [B, H, nB, D]."""
    B, H = bits["q"].shape[:2]
    qp, kp = [], []
    for b in range(B):
        qrow, krow = [], []
        for h in range(H):
            qrow.append(oracle.pool_blocks(oracle.bf16_bits_to_f64(bits["q"][b, h]), block))
            krow.append(oracle.pool_blocks(oracle.bf16_bits_to_f64(bits["k"][b, h]), block))
        qp.append(qrow)
        kp.append(krow)
    return np.array(qp), np.array(kp)


def oracle_select(wl: workloads.Workload, scores: np.ndarray, keep_ratio=None):
    nb = scores.shape[-1]
    if wl.mode == "mass":
        forced = (oracle.first_frame_blocks(wl.grid_h, wl.grid_w, wl.block, nb)
                  if wl.force_first_frame else [])
        cap = oracle.mass_cap(nb, wl.max_keep_ratio, len(forced))
        kept = oracle.select_cummass(scores, wl.mass_threshold, cap, forced)
        return kept, dict(mode="mass", tau=wl.mass_threshold, forced=forced, k=0, cap=cap)
    r = wl.keep_ratio if keep_ratio is None else keep_ratio
    k = oracle.topk_count(nb, r, wl.topk if keep_ratio is None else 0)
    kept = oracle.select_topk(scores, k)
    return kept, dict(mode="topk", k=k, forced=[], tau=0.0, cap=k)


def flat_rows(kept):
    """Nested [B][H][nB] kept lists -> flat list of lists."""
    return [row for b in kept for h in b for row in h]


def scale_of(wl) -> float:
    return 1.0 / math.sqrt(wl.head_dim)
