"""CPU oracle for block-sparse video self-attention -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The GPU library never calls it, and it shares no code with the
GPU path: every function here is a plain, slow, float64 restatement of what the
path computes, written for a reader to check by eye.

The fused QKNorm + RoPE + pool producer (Section 4.2.5 names "fused RoPE +
norm"; Appendix A.2.2 lists fused QKNorm+RoPE in the LTX-2.3 stack) is in
qknorm_rope.py with its own readings; feat_norm token pruning (Section 4.2.3;
Appendix A.2.2 keeps 50% of video tokens by that score) in token_prune.py;
8-bit attention (Section 4.2.4 points to the SageAttention series) in
fp8_attention.py; the first-order remainder of non-kept blocks (Section 4.2.2)
in remainder.py.

What the paper fixes (Section 4.2.2, "Sparse Attention"; Appendix A.2.2, the
LTX-2.3 pipeline): attention over the spatiotemporal token set is replaced by a
block-sparse pattern; blocks are routed by a score ("score-based routing", a
"block-wise similarity metric"); the blocks that are kept ("critical blocks")
are computed exactly; block size 64 and density 0.1 in the LTX-2.3 setting; a
dense FlashAttention fallback.  The paper prints no formula for the routing
score or the selection rule, so this oracle takes the readings listed in the
design notes (mean-pooled block summaries, scaled dot-product block score,
top-k or cumulative-softmax-mass selection, non-kept blocks contribute nothing).

Parity status per function:
  blocks.pool_blocks          pinned (closed form on arithmetic progressions, brute force)
  select.block_scores         pinned (brute force, transposition-sensitive)
  select.select_topk          pinned (brute-force sort with index tie-break, hand-worked fixture)
  select.select_cummass       pinned (independent cumsum search, closed forms, invariants)
  attention.block_sparse_attention / dense_attention
                              pinned (pure-Python brute force, torch SDPA in float64,
                                      closed forms, invariants)
  qknorm_rope.round_bf16      pinned (bit-level float32 rounding, ties, double-rounding case)
  qknorm_rope.rms_norm        pinned (closed forms, library norm, scale invariance)
  qknorm_rope.rope_angles / apply_rope
                              pinned (hand-derived angles, complex multiplication,
                                      identity at the origin, norm, relative position)
  qknorm_rope.qknorm_rope_pool
                              pinned (pool of the rounded outputs; parts above)
  token_prune.token_scores    pinned (library norm, closed forms, axis check)
  token_prune.select_tokens   pinned (pure-Python sort with tie key, hand-worked example)
  token_prune.keep_count      pinned (closed forms incl. the 0.1*1180 case)
  token_prune.gather_tokens / scatter_tokens
                              pinned (round trip, placement and base identities)
  fp8_attention.round_e4m3 / e4m3_value / encode_e4m3
                              pinned (format code table, brute-force nearest-even
                                      search, library float32 cast)
  fp8_attention.scale_exponent / quantize_qkv
                              pinned (brute-force exponents, pure-Python grouping
                                      and codes, error bounds)
  fp8_attention.fp8_block_sparse_attention
                              pinned (smoothing invariance, exactly representable
                                      inputs equal plain attention)
  remainder.block_moments     pinned (brute force over tokens, independent identity)
  remainder.remainder_attention
                              pinned (term-by-term sum over dropped tokens,
                                      exact on constant-key blocks, dense when
                                      all kept, constant values, convergence
                                      orders: second in the key deviations for
                                      the plain expansion, first for the
                                      block-mean form where queries vary)
  The paper's own routing rule and its formula for the first-order remainder of
  non-kept blocks: parity unpinned (neither is written out in the paper's text;
  remainder.py implements the plain first-order expansion about the block-mean
  keys, and the block-mean-query form the kernels compute).
"""
from .blocks import bf16_bits_to_f64, num_blocks, block_bounds, pool_blocks
from .select import (block_scores, topk_count, select_topk, first_frame_blocks,
                     mass_cap, select_cummass, kept_to_arrays, kept_to_mask)
from .attention import block_sparse_attention, dense_attention
from .qknorm_rope import (round_bf16, rms_norm, rope_pair_groups, rope_angles, apply_rope,
                          norm_rope, qknorm_rope_pool)
from .token_prune import token_scores, keep_count, select_tokens, gather_tokens, scatter_tokens
from .fp8_attention import (e4m3_value, round_e4m3, encode_e4m3, scale_exponent, quantize_qkv,
                            fp8_block_sparse_attention)

__all__ = [
    "bf16_bits_to_f64", "num_blocks", "block_bounds", "pool_blocks",
    "block_scores", "topk_count", "select_topk", "first_frame_blocks", "mass_cap",
    "select_cummass", "kept_to_arrays", "kept_to_mask",
    "block_sparse_attention", "dense_attention",
    "round_bf16", "rms_norm", "rope_pair_groups", "rope_angles", "apply_rope", "norm_rope",
    "qknorm_rope_pool", "token_scores", "keep_count", "select_tokens", "gather_tokens",
    "e4m3_value", "round_e4m3", "encode_e4m3", "scale_exponent", "quantize_qkv",
    "fp8_block_sparse_attention",
    "scatter_tokens",
]
