"""Block-sparse spatiotemporal self-attention for video DiTs on MI355X (gfx950).

The compute path is libsva.so (HIP kernels behind the C ABI in include/sva.h);
this package is its Python binding plus the synthetic-input generator and the
workload shapes.  Importing the package does not load the library; the first
call into it does, and raises if libsva.so has not been built.
"""
from . import workloads
from ._lib import (SvaError, Problem, SelectParams, RopeParams, load, problem, problem_for,
                   select_topk, select_mass, select_for, num_blocks, max_keep, pool_blocks,
                   qknorm_rope_pool, select_blocks, sparse_attention, dense_attention,
                   status_string, LIB_PATH, Tokens, tokens, token_keep_count, token_select, token_select_noalloc,
                   token_gather, token_scatter, token_select_workspace, Fp8Tensors, fp8_padded_len, fp8_code_dim,
                   quantize_fp8, sparse_attention_fp8, dense_attention_fp8, remainder_workspace,
                   block_moments, sparse_attention_remainder)

__all__ = [
    "workloads", "SvaError", "Problem", "SelectParams", "RopeParams", "load", "problem",
    "problem_for", "select_topk", "select_mass", "select_for", "num_blocks", "max_keep",
    "pool_blocks", "qknorm_rope_pool", "select_blocks", "sparse_attention", "dense_attention",
    "status_string", "LIB_PATH", "Tokens", "tokens", "token_keep_count", "token_select", "token_select_noalloc",
    "token_gather", "token_scatter", "token_select_workspace", "Fp8Tensors", "fp8_padded_len", "fp8_code_dim",
    "quantize_fp8", "sparse_attention_fp8", "dense_attention_fp8", "remainder_workspace",
    "block_moments", "sparse_attention_remainder",
]
