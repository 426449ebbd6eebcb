"""C-ABI checks that need no GPU: libsva.so loads, exports every function
include/sva.h declares, derives block counts and kept-block bounds on the host,
and rejects bad arguments with the documented status before any launch.

Compute entry points are called here only with arguments that fail validation
(null or misaligned pointers, bad shapes), which return before any HIP call.
"""
import ctypes

import pytest

import paper_2606_23743_amd as sva
from paper_2606_23743_amd import _lib, workloads

pytestmark = pytest.mark.cpu


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_every_declared_symbol_is_exported(lib):
    names = _lib.header_functions()
    assert set(names) >= {"sva_pool_blocks", "sva_select_blocks", "sva_sparse_attention",
                          "sva_dense_attention", "sva_num_blocks", "sva_max_keep",
                          "sva_qknorm_rope_pool", "sva_token_keep_count", "sva_token_select",
                          "sva_token_select_workspace", "sva_fp8_padded_len", "sva_fp8_code_dim", "sva_quantize_fp8",
                          "sva_sparse_attention_fp8", "sva_dense_attention_fp8",
                          "sva_token_gather", "sva_token_scatter", "sva_status_string",
                          "sva_remainder_workspace", "sva_remainder_workspace_heads", "sva_block_moments",
                          "sva_sparse_attention_remainder",
                          "sva_version"}
    for n in names:
        assert hasattr(lib, n), n


def test_library_binds_every_symbol_at_load():
    """Immediate binding: a kernel launch stub or any other symbol left
    undefined fails here instead of at its first call."""
    import os
    ctypes.CDLL(_lib.LIB_PATH, mode=os.RTLD_NOW | os.RTLD_LOCAL)


def test_version_and_status_strings(lib):
    assert lib.sva_version() == 1
    for st in range(6):
        assert _lib.status_string(st) not in ("", "unknown status")
    assert _lib.status_string(99) == "unknown status"


@pytest.mark.parametrize("wl,nb", [(workloads.TINY, 16), (workloads.SMALL_2B, 512),
                                   (workloads.MID_22B, 989), (workloads.LARGE_64B, 872),
                                   (workloads.CFG_SWEEP, 1182)])
def test_num_blocks(wl, nb):
    assert sva.num_blocks(sva.problem_for(wl)) == nb


def test_max_keep_per_workload():
    assert sva.max_keep(sva.problem_for(workloads.TINY), sva.select_for(workloads.TINY)) == 4
    assert sva.max_keep(sva.problem_for(workloads.SMALL_2B), sva.select_for(workloads.SMALL_2B)) == 128
    assert sva.max_keep(sva.problem_for(workloads.MID_22B), sva.select_for(workloads.MID_22B)) == 297
    assert sva.max_keep(sva.problem_for(workloads.LARGE_64B), sva.select_for(workloads.LARGE_64B)) == 131
    p = sva.problem_for(workloads.CFG_SWEEP)
    assert [sva.max_keep(p, sva.select_topk(r)) for r in (1.0, 0.5, 0.25, 0.1)] == [1182, 591, 296, 119]
    # the count epsilon: 0.1 * 1180 is a hair above 118 in binary64
    p = sva.problem(1, 1, 1180 * 64, 64, (1, 1, 1180 * 64), 64)
    assert sva.max_keep(p, sva.select_topk(0.1)) == 118
    # cap never below the forced first-frame blocks: 34*60 tokens per frame -> 32 blocks
    pm = sva.problem_for(workloads.MID_22B)
    assert sva.max_keep(pm, sva.select_mass(0.9, 0.01, True)) == 32
    assert sva.max_keep(pm, sva.select_mass(0.9, 0.01, False)) == 10


def _status(fn, *args):
    return fn(*args)


def test_problem_validation(lib):
    out = ctypes.c_int32()
    good = sva.problem_for(workloads.TINY)
    assert lib.sva_num_blocks(ctypes.byref(good), ctypes.byref(out)) == _lib.SVA_OK
    assert lib.sva_num_blocks(None, ctypes.byref(out)) == _lib.SVA_ERR_INVALID_ARG
    assert lib.sva_num_blocks(ctypes.byref(good), None) == _lib.SVA_ERR_INVALID_ARG
    bad_grid = sva.problem(1, 2, 1024, 64, (4, 16, 15), 64)
    assert lib.sva_num_blocks(ctypes.byref(bad_grid), ctypes.byref(out)) == _lib.SVA_ERR_SHAPE
    bad_d = sva.problem(1, 2, 1024, 96, (4, 16, 16), 64)
    assert lib.sva_num_blocks(ctypes.byref(bad_d), ctypes.byref(out)) == _lib.SVA_ERR_UNSUPPORTED
    bad_s = sva.problem(1, 2, 1024, 64, (4, 16, 16), 32)
    assert lib.sva_num_blocks(ctypes.byref(bad_s), ctypes.byref(out)) == _lib.SVA_ERR_UNSUPPORTED
    zero_b = sva.problem(0, 2, 1024, 64, (4, 16, 16), 64)
    assert lib.sva_num_blocks(ctypes.byref(zero_b), ctypes.byref(out)) == _lib.SVA_ERR_INVALID_ARG
    bad_dt = sva.problem(1, 2, 1024, 64, (4, 16, 16), 64)
    bad_dt.out_dtype = 7
    assert lib.sva_num_blocks(ctypes.byref(bad_dt), ctypes.byref(out)) == _lib.SVA_ERR_INVALID_ARG
    nan_scale = sva.problem(1, 2, 1024, 64, (4, 16, 16), 64, softmax_scale=float("nan"))
    assert lib.sva_num_blocks(ctypes.byref(nan_scale), ctypes.byref(out)) == _lib.SVA_ERR_INVALID_ARG
    huge = sva.problem(40000, 40000, 4096, 64, (1, 64, 64), 64)
    assert lib.sva_num_blocks(ctypes.byref(huge), ctypes.byref(out)) == _lib.SVA_ERR_SHAPE


def test_select_param_validation(lib):
    out = ctypes.c_int32()
    p = sva.problem_for(workloads.TINY)
    for sel, want in [(sva.select_topk(0.0, 0), _lib.SVA_ERR_INVALID_ARG),
                      (sva.select_topk(1.5, 0), _lib.SVA_ERR_INVALID_ARG),
                      (sva.select_topk(0.5, -1), _lib.SVA_ERR_INVALID_ARG),
                      (sva.select_mass(0.0, 0.3, True), _lib.SVA_ERR_INVALID_ARG),
                      (sva.select_mass(0.9, 1.5, True), _lib.SVA_ERR_INVALID_ARG),
                      (_lib.SelectParams(7, 0.5, 0, 0, 0, 0), _lib.SVA_ERR_INVALID_ARG),
                      (sva.select_topk(0.0, 99), _lib.SVA_OK)]:
        assert lib.sva_max_keep(ctypes.byref(p), ctypes.byref(sel), ctypes.byref(out)) == want
    assert out.value == 16    # topk clamped to nB


def test_compute_entry_points_reject_before_launch(lib):
    p = sva.problem_for(workloads.TINY)
    sel = sva.select_for(workloads.TINY)
    A = 1 << 20          # a fake, 16-byte aligned address: never dereferenced on these paths
    assert lib.sva_pool_blocks(ctypes.byref(p), None, A, A, A, None) == _lib.SVA_ERR_INVALID_ARG
    assert lib.sva_pool_blocks(ctypes.byref(p), A + 2, A, A, A, None) == _lib.SVA_ERR_ALIGNMENT
    assert lib.sva_pool_blocks(None, A, A, A, A, None) == _lib.SVA_ERR_INVALID_ARG
    assert lib.sva_select_blocks(ctypes.byref(p), ctypes.byref(sel), A, A, 3, A, A, None, None) \
        == _lib.SVA_ERR_SHAPE                                    # kmax 3 < k = 4
    assert lib.sva_select_blocks(ctypes.byref(p), ctypes.byref(sel), A, None, 4, A, A, None, None) \
        == _lib.SVA_ERR_INVALID_ARG
    assert lib.sva_select_blocks(ctypes.byref(p), ctypes.byref(sel), A, A + 1, 4, A, A, None, None) \
        == _lib.SVA_ERR_ALIGNMENT
    big = sva.problem(1, 1, 2049 * 64, 64, (1, 1, 2049 * 64), 64)
    assert lib.sva_select_blocks(ctypes.byref(big), ctypes.byref(sel), A, A, 4, A, A, None, None) \
        == _lib.SVA_ERR_UNSUPPORTED                              # nB above the register bound
    assert lib.sva_sparse_attention(ctypes.byref(p), A, A, A, A, A, 0, A, None, None) == _lib.SVA_ERR_SHAPE
    assert lib.sva_sparse_attention(ctypes.byref(p), A, A, None, A, A, 4, A, None, None) \
        == _lib.SVA_ERR_INVALID_ARG
    assert lib.sva_sparse_attention(ctypes.byref(p), A, A, A, A, A, 4, A + 8, None, None) \
        == _lib.SVA_ERR_ALIGNMENT
    assert lib.sva_dense_attention(ctypes.byref(p), A, A, A, None, None, None) == _lib.SVA_ERR_INVALID_ARG
    assert lib.sva_dense_attention(ctypes.byref(p), A, A, A, A, A + 2, None) == _lib.SVA_ERR_ALIGNMENT


def _remainder_bytes(B, H, N, D, S):
    up = lambda x: (x + 255) // 256 * 256
    nb = -(-N // S)
    nbp = (nb + 31) // 32 * 32
    nbr = (nb + 255) // 256 * 256            # rows of each 32-key chunk of the weights
    bh = B * H
    return (up(bh * N * D * 4) + up(bh * N * 4) + 2 * up(bh * nbp * D * 2) + 2 * up(bh * nbp * D * D * 2)
            + up(bh * nbp * nbr * 2) + up(bh * nbp * 4))


def test_remainder_workspace_and_rejects_before_launch(lib):
    for wl in (workloads.TINY, workloads.LARGE_64B, workloads.MID_22B):
        p = sva.problem_for(wl)
        ws = ctypes.c_size_t(0)
        assert lib.sva_remainder_workspace(ctypes.byref(p), ctypes.byref(ws)) == _lib.SVA_OK
        assert ws.value == _remainder_bytes(wl.batch, wl.heads, wl.seq_len, wl.head_dim, wl.block)
        # passes of fewer (batch, head) pairs: the same layout for that many
        for g in (1, 2, wl.batch * wl.heads):
            assert lib.sva_remainder_workspace_heads(ctypes.byref(p), g, ctypes.byref(ws)) == _lib.SVA_OK
            assert ws.value == _remainder_bytes(1, g, wl.seq_len, wl.head_dim, wl.block), (wl.name, g)
        for g in (0, -1, wl.batch * wl.heads + 1):
            assert lib.sva_remainder_workspace_heads(ctypes.byref(p), g, ctypes.byref(ws)) == _lib.SVA_ERR_SHAPE
        assert lib.sva_remainder_workspace_heads(ctypes.byref(p), 1, None) == _lib.SVA_ERR_INVALID_ARG
    p = sva.problem_for(workloads.TINY)
    need = ctypes.c_size_t(0)
    lib.sva_remainder_workspace_heads(ctypes.byref(p), 1, ctypes.byref(need))   # the least the call takes
    A = 1 << 20
    f = lib.sva_sparse_attention_remainder
    assert lib.sva_remainder_workspace(ctypes.byref(p), None) == _lib.SVA_ERR_INVALID_ARG
    assert f(ctypes.byref(p), A, A, A, None, A, A, A, 4, A, need.value, A, None, None) == _lib.SVA_ERR_INVALID_ARG
    assert f(ctypes.byref(p), A, A, A, A, A, A, A, 0, A, need.value, A, None, None) == _lib.SVA_ERR_SHAPE
    assert f(ctypes.byref(p), A, A, A, A, A, A, A, 4, A, need.value - 1, A, None, None) == _lib.SVA_ERR_SHAPE
    assert f(ctypes.byref(p), A, A, A, A, A, A, A, 4, A + 16, need.value, A, None, None) == _lib.SVA_ERR_ALIGNMENT
    assert f(ctypes.byref(p), A, A, A, A + 4, A, A, A, 4, A, need.value, A, None, None) == _lib.SVA_ERR_ALIGNMENT
    big = sva.problem(1, 1, 4097 * 64, 64, (1, 1, 4097 * 64), 64)
    assert lib.sva_remainder_workspace(ctypes.byref(big), ctypes.byref(need)) == _lib.SVA_ERR_UNSUPPORTED
    assert f(ctypes.byref(big), A, A, A, A, A, A, A, 4, A, 1 << 40, A, None, None) == _lib.SVA_ERR_UNSUPPORTED
    assert lib.sva_block_moments(ctypes.byref(p), A, A, A, None, A, None) == _lib.SVA_ERR_INVALID_ARG
    assert lib.sva_block_moments(ctypes.byref(p), A, A, A, A + 2, A, None) == _lib.SVA_ERR_ALIGNMENT
    assert lib.sva_block_moments(ctypes.byref(big), A, A, A, A, A, None) == _lib.SVA_ERR_UNSUPPORTED


def test_qknorm_rope_pool_rejects_before_launch(lib):
    p = sva.problem_for(workloads.TINY)
    A = 1 << 20
    B = A + (1 << 24)    # disjoint from A for this problem's 256 KB tensors
    ok = _lib.RopeParams(1e-6, 10000.0)
    f = lib.sva_qknorm_rope_pool
    assert f(ctypes.byref(p), None, A, A, A, A, B, B, A, A, None) == _lib.SVA_ERR_INVALID_ARG
    assert f(ctypes.byref(p), ctypes.byref(ok), None, A, A, A, B, B, A, A, None) == _lib.SVA_ERR_INVALID_ARG
    for bad in (_lib.RopeParams(-1.0, 10000.0), _lib.RopeParams(1e-6, 1.0),
                _lib.RopeParams(float("nan"), 10000.0), _lib.RopeParams(1e-6, float("inf"))):
        assert f(ctypes.byref(p), ctypes.byref(bad), A, A, A, A, B, B, A, A, None) == _lib.SVA_ERR_INVALID_ARG
    assert f(ctypes.byref(p), ctypes.byref(ok), A + 2, A, A, A, B, B, A, A, None) == _lib.SVA_ERR_ALIGNMENT
    assert f(ctypes.byref(p), ctypes.byref(ok), A, A, A + 1, A, B, B, A, A, None) == _lib.SVA_ERR_ALIGNMENT
    # an output that overlaps its input without being it
    assert f(ctypes.byref(p), ctypes.byref(ok), A, A, A, A, A + 64, B, A, A, None) == _lib.SVA_ERR_INVALID_ARG
    assert f(None, ctypes.byref(ok), A, A, A, A, B, B, A, A, None) == _lib.SVA_ERR_INVALID_ARG


def test_token_keep_count_matches_the_oracle_reading():
    import oracle.token_prune as otp
    for n, r in ((111600, 0.5), (1180, 0.1), (10, 0.25), (7, 1e-9), (7, 1.0), (3, 0.34)):
        assert sva.token_keep_count(sva.tokens(2, n, 8), r) == otp.keep_count(n, r), (n, r)


def test_token_entry_points_reject_before_launch(lib):
    A = 1 << 20
    B = A + (1 << 26)
    t = sva.tokens(2, 100, 64)
    k = ctypes.c_int32()
    for bad in (sva.tokens(0, 100, 64), sva.tokens(1, 0, 64), sva.tokens(1, 100, 4), sva.tokens(1, 100, 12)):
        assert lib.sva_token_keep_count(ctypes.byref(bad), 0.5, ctypes.byref(k)) == _lib.SVA_ERR_INVALID_ARG
    assert lib.sva_token_keep_count(ctypes.byref(sva.tokens(1 << 16, 1 << 16, 8)), 0.5, ctypes.byref(k)) \
        == _lib.SVA_ERR_SHAPE                                    # B*N beyond int32
    for r in (0.0, -0.5, 1.0000001, float("nan")):
        assert lib.sva_token_keep_count(ctypes.byref(t), r, ctypes.byref(k)) == _lib.SVA_ERR_INVALID_ARG
    assert lib.sva_token_keep_count(ctypes.byref(t), 0.5, None) == _lib.SVA_ERR_INVALID_ARG
    ws = ctypes.c_size_t()
    assert lib.sva_token_select_workspace(ctypes.byref(t), ctypes.byref(ws)) == _lib.SVA_OK
    assert ws.value == 2 * 33024 and sva.token_select_workspace(t) == ws.value
    assert lib.sva_token_select_workspace(ctypes.byref(t), None) == _lib.SVA_ERR_INVALID_ARG
    W = ws.value
    sel = lib.sva_token_select
    assert sel(ctypes.byref(t), 0.5, None, A, A, A, B, W, None) == _lib.SVA_ERR_INVALID_ARG
    assert sel(ctypes.byref(t), 0.5, A, A, A, A, None, W, None) == _lib.SVA_ERR_INVALID_ARG
    assert sel(ctypes.byref(t), 0.5, A, A, A, A, B, W - 1, None) == _lib.SVA_ERR_SHAPE
    assert sel(ctypes.byref(t), 0.5, A + 8, A, A, A, B, W, None) == _lib.SVA_ERR_ALIGNMENT
    assert sel(ctypes.byref(t), 0.5, A, A + 4, A, A, B, W, None) == _lib.SVA_ERR_ALIGNMENT
    assert sel(ctypes.byref(t), 0.5, A, A, A, A, B + 4, W, None) == _lib.SVA_ERR_ALIGNMENT
    assert sel(ctypes.byref(t), 2.0, A, A, A, A, B, W, None) == _lib.SVA_ERR_INVALID_ARG
    # the allocation-free form: the same checks, and more than 16 batch
    # entries (its static workspace) rejected, all before any device call
    nsel = lib.sva_token_select_noalloc
    assert nsel(ctypes.byref(t), 0.5, None, A, A, A, None) == _lib.SVA_ERR_INVALID_ARG
    assert nsel(ctypes.byref(t), 0.5, A, A, A, None, None) == _lib.SVA_ERR_INVALID_ARG
    assert nsel(ctypes.byref(t), 0.5, A + 8, A, A, A, None) == _lib.SVA_ERR_ALIGNMENT
    assert nsel(ctypes.byref(t), 2.0, A, A, A, A, None) == _lib.SVA_ERR_INVALID_ARG
    assert nsel(ctypes.byref(sva.tokens(17, 100, 64)), 0.5, A, A, A, A, None) == _lib.SVA_ERR_SHAPE
    g = lib.sva_token_gather
    assert g(ctypes.byref(t), 0, A, A, B, None) == _lib.SVA_ERR_SHAPE
    assert g(ctypes.byref(t), 101, A, A, B, None) == _lib.SVA_ERR_SHAPE
    assert g(ctypes.byref(t), 50, A, None, B, None) == _lib.SVA_ERR_INVALID_ARG
    assert g(ctypes.byref(t), 50, A, A + 2, B, None) == _lib.SVA_ERR_ALIGNMENT
    sc = lib.sva_token_scatter
    assert sc(ctypes.byref(t), 50, A, A, B, None, None) == _lib.SVA_ERR_INVALID_ARG
    assert sc(ctypes.byref(t), 50, A + 8, A, B, B, None) == _lib.SVA_ERR_ALIGNMENT
    # out overlapping y_kept, and a base that overlaps out without being it
    assert sc(ctypes.byref(t), 50, A, A, B, A + 256, None) == _lib.SVA_ERR_INVALID_ARG
    assert sc(ctypes.byref(t), 50, A, A, B + 256, B, None) == _lib.SVA_ERR_INVALID_ARG
    assert sc(None, 50, A, A, B, B, None) == _lib.SVA_ERR_INVALID_ARG


def test_fp8_entry_points_reject_before_launch(lib):
    p = sva.problem_for(workloads.TINY)                       # D=64, S=64
    n = ctypes.c_int32()
    assert lib.sva_fp8_padded_len(ctypes.byref(p), ctypes.byref(n)) == _lib.SVA_OK and n.value == 1024
    p112 = sva.problem_for(workloads.SMALL_2B)                # D=112: carried as 128 code channels
    assert lib.sva_fp8_padded_len(ctypes.byref(p112), ctypes.byref(n)) == _lib.SVA_OK and n.value == 512 * 64
    assert lib.sva_fp8_code_dim(ctypes.byref(p112), ctypes.byref(n)) == _lib.SVA_OK and n.value == 128
    assert lib.sva_fp8_code_dim(ctypes.byref(p), ctypes.byref(n)) == _lib.SVA_OK and n.value == 64
    assert lib.sva_fp8_code_dim(ctypes.byref(p), None) == _lib.SVA_ERR_INVALID_ARG
    assert lib.sva_fp8_padded_len(ctypes.byref(p), None) == _lib.SVA_ERR_INVALID_ARG
    A = 1 << 20
    ok = _lib.Fp8Tensors(A, A, A, A, A, A, A)
    f = lib.sva_quantize_fp8
    assert f(ctypes.byref(p), A, A, A, None, None) == _lib.SVA_ERR_INVALID_ARG
    assert f(ctypes.byref(p), A, A, None, ctypes.byref(ok), None) == _lib.SVA_ERR_INVALID_ARG
    assert f(ctypes.byref(p), A, A, A, ctypes.byref(_lib.Fp8Tensors(A, A, A, A, A, A, None)), None) \
        == _lib.SVA_ERR_INVALID_ARG                           # k_mean is written by the quantiser
    assert f(ctypes.byref(p), A, A, A, ctypes.byref(_lib.Fp8Tensors(A + 8, A, A, A, A, A, A)), None) \
        == _lib.SVA_ERR_ALIGNMENT
    assert f(ctypes.byref(p), A + 2, A, A, ctypes.byref(ok), None) == _lib.SVA_ERR_ALIGNMENT
    g = lib.sva_sparse_attention_fp8
    assert g(ctypes.byref(p), ctypes.byref(ok), A, A, 0, A, None, None) == _lib.SVA_ERR_SHAPE
    assert g(ctypes.byref(p), ctypes.byref(ok), A, A, 2048, A, None, None) == _lib.SVA_ERR_UNSUPPORTED
    assert g(ctypes.byref(p), ctypes.byref(ok), None, A, 4, A, None, None) == _lib.SVA_ERR_INVALID_ARG
    assert g(ctypes.byref(p), ctypes.byref(ok), A, A, 4, A + 8, None, None) == _lib.SVA_ERR_ALIGNMENT
    assert g(ctypes.byref(p), ctypes.byref(_lib.Fp8Tensors(A, A, A, A + 2, A, A, None)), A, A, 4, A, None,
             None) == _lib.SVA_ERR_ALIGNMENT
    h = lib.sva_dense_attention_fp8
    assert h(ctypes.byref(p), None, A, None, None) == _lib.SVA_ERR_INVALID_ARG
    assert h(ctypes.byref(sva.problem(1, 1, 2048 * 64, 64, (1, 1, 2048 * 64), 64)), ctypes.byref(ok), A, None,
             None) == _lib.SVA_ERR_UNSUPPORTED                # nB = 2048 above the list bound
