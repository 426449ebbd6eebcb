"""Workload shapes for block-sparse video self-attention.

Each workload is one video-DiT self-attention layer: Q/K/V of shape [B, H, N, D]
over a T x H x W latent token grid flattened t-major, a block size S (query block
== key block), and a block-selection rule.  The shapes follow the paper's model
families (Section 5, Table 1; Appendix A.2: LTX-2.3 stage 2 at 1088x1920 and 241
frames, SANA-Video at 832x480 and 81 frames) and the sparse-attention settings of
Appendix A.2.2 (block 64, density 0.1).

This module is data only: sizes and selection parameters.  It holds none of the
method's arithmetic (block counts, k from a ratio, caps) -- the kernels' host
code and the oracle each derive those themselves.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    heads: int
    head_dim: int
    grid_t: int
    grid_h: int
    grid_w: int
    block: int
    mode: str                      # "topk" | "mass"
    keep_ratio: float = 0.0        # top-k: fraction of KV blocks kept per query block
    topk: int = 0                  # top-k: explicit count (overrides keep_ratio when > 0)
    mass_threshold: float = 0.0    # mass: cumulative softmax mass to reach
    max_keep_ratio: float = 1.0    # mass: cap on kept blocks as a fraction of all blocks
    force_first_frame: bool = False
    sink_tokens: int = 0           # keys of the first sink_tokens tokens are scaled ...
    sink_scale: float = 1.0        # ... by sink_scale (attention-sink structure)
    ratios: Tuple[float, ...] = field(default_factory=tuple)  # extra keep ratios (sweep)
    seed: int = 0

    @property
    def seq_len(self) -> int:
        return self.grid_t * self.grid_h * self.grid_w

    def with_ratio(self, r: float) -> "Workload":
        return replace(self, keep_ratio=float(r), topk=0, ratios=())


# Seeds: 20260000 + workload number.
TINY = Workload("tiny_plumbing_b1h2d64_n1024", 1, 2, 64, 4, 16, 16, 64, "topk",
                topk=4, seed=20260001)
SMALL_2B = Workload("small_2b_b1h20d112_n32760", 1, 20, 112, 21, 30, 52, 64, "topk",
                    keep_ratio=0.25, seed=20260002)
MID_22B = Workload("mid_22b_b1h32d128_n63240_mass", 1, 32, 128, 31, 34, 60, 64, "mass",
                   mass_threshold=0.9, max_keep_ratio=0.30, force_first_frame=True,
                   seed=20260003)
LARGE_64B = Workload("large_64b_b1h48d128_n111600_s128", 1, 48, 128, 31, 45, 80, 128, "topk",
                     keep_ratio=0.15, sink_tokens=256, sink_scale=3.0, seed=20260004)
CFG_SWEEP = Workload("cfg_sweep_b2h24d128_n75600", 2, 24, 128, 21, 45, 80, 64, "topk",
                     keep_ratio=0.25, ratios=(1.0, 0.5, 0.25, 0.1), seed=20260005)

ALL = (TINY, SMALL_2B, MID_22B, LARGE_64B, CFG_SWEEP)
BY_NAME = {w.name: w for w in ALL}


def small_case(name: str, batch: int, heads: int, head_dim: int, grid: Tuple[int, int, int],
               block: int, mode: str = "topk", seed: int = 1, **kw) -> Workload:
    """A reduced workload for parity tests (sizes the oracle finishes in seconds)."""
    t, h, w = grid
    return Workload(name, batch, heads, head_dim, t, h, w, block, mode, seed=seed, **kw)


def find(name: str) -> Optional[Workload]:
    return BY_NAME.get(name)
