"""Token blocks and block mean-pooling (oracle; test infrastructure only).

Reading of the paper (Section 4.2.2; Appendix A.2.2 "block size is 64"): the
spatiotemporal token grid T x H x W is flattened t-major (n = (t*H + y)*W + x)
and cut into contiguous blocks of S tokens; the last block may be partial.  A
block's summary is the mean of its valid tokens (a partial block is averaged
over the tokens it has, not over S).
"""
from __future__ import annotations

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Decode bf16 bit patterns (uint16) to float64 exactly.

    A bf16 value is the upper half of an IEEE binary32 value, so placing the 16
    bits above 16 zero bits gives the same number as a float32, which widens to
    float64 without rounding.
    """
    bits = np.asarray(bits, dtype=np.uint16)
    as32 = bits.astype(np.uint32) << np.uint32(16)
    return as32.view(np.float32).astype(np.float64)


def num_blocks(seq_len: int, block: int) -> int:
    """Number of blocks: ceil(N / S)."""
    return -(-int(seq_len) // int(block))


def block_bounds(seq_len: int, block: int):
    """[(start, stop)] of every block; stop of the last block is clipped to N."""
    return [(i * block, min((i + 1) * block, seq_len)) for i in range(num_blocks(seq_len, block))]


def pool_blocks(x: np.ndarray, block: int) -> np.ndarray:
    """Mean over the valid tokens of each block.

    x: float64 [..., N, D]  ->  [..., nB, D]
    """
    x = np.asarray(x, dtype=np.float64)
    n = x.shape[-2]
    bounds = block_bounds(n, block)
    out = np.empty(x.shape[:-2] + (len(bounds), x.shape[-1]), dtype=np.float64)
    for i, (a, b) in enumerate(bounds):
        out[..., i, :] = x[..., a:b, :].sum(axis=-2) / (b - a)
    return out
