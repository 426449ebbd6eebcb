"""GPU parity on reduced shapes: every step of the HIP path against the oracle,
element by element, over every head dim (64, 112, 128) and block size (64, 128),
both selection rules, ragged tails, a sequence shorter than one block, and the
degenerate index lists (empty rows, out-of-range entries, duplicates, unsorted).
"""
import math

import numpy as np
import pytest

import oracle
import paper_2606_23743_amd as sva
from paper_2606_23743_amd import inputs, workloads

from . import parity
from .gpu_cases import (device_inputs, flat_rows, oracle_pool_all, oracle_select, say, scale_of)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SC = workloads.small_case
CASES = [
    SC("d64_s64_topk", 2, 3, 64, (3, 10, 13), 64, "topk", keep_ratio=0.5, seed=101),
    SC("d112_s64_topk", 1, 3, 112, (3, 10, 13), 64, "topk", keep_ratio=0.3, seed=102),
    SC("d128_s64_mass", 2, 2, 128, (5, 8, 9), 64, "mass", mass_threshold=0.9,
       max_keep_ratio=0.5, force_first_frame=True, seed=103),
    SC("d128_s128_topk", 1, 3, 128, (4, 10, 13), 128, "topk", keep_ratio=0.5, seed=104),
    SC("d112_s128_mass", 1, 2, 112, (6, 9, 11), 128, "mass", mass_threshold=0.8,
       max_keep_ratio=0.6, force_first_frame=False, seed=105),
    SC("d64_s128_topk", 2, 2, 64, (4, 10, 13), 128, "topk", topk=2, seed=106),
    SC("d128_s64_single_partial_block", 1, 2, 128, (1, 5, 7), 64, "topk", topk=1, seed=107),
    SC("d128_s64_exact_multiple", 1, 2, 128, (2, 8, 16), 64, "topk", keep_ratio=0.5, seed=108),
    SC("d128_s64_sink", 1, 2, 128, (4, 12, 16), 64, "topk", keep_ratio=0.25, sink_tokens=128,
       sink_scale=3.0, seed=109),
    workloads.TINY,
]

_cache = {}


def run_case(wl):
    if wl.name in _cache:
        return _cache[wl.name]
    say(f"[case {wl.name}] B={wl.batch} H={wl.heads} N={wl.seq_len} D={wl.head_dim} S={wl.block}")
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    sel = sva.select_for(wl)
    nb = sva.num_blocks(prob)
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    kv_idx, kv_count, mask = sva.select_blocks(prob, sel, qp, kp, want_mask=True)
    out, lse = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], kv_idx, kv_count, want_lse=True)
    dout, dlse = sva.dense_attention(prob, dev["q"], dev["k"], dev["v"], want_lse=True)
    torch.cuda.synchronize()
    g = dict(qp=qp.cpu().numpy(), kp=kp.cpu().numpy(), idx=kv_idx.cpu().numpy(),
             cnt=kv_count.cpu().numpy(), mask=mask.cpu().numpy(), out=out.float().cpu().numpy(),
             lse=lse.cpu().numpy(), dout=dout.float().cpu().numpy(), dlse=dlse.cpu().numpy())
    # oracle on the same bytes
    oqp, okp = oracle_pool_all(bits, wl.block)
    scores = oracle.block_scores(oqp, okp, scale_of(wl))
    kept, info = oracle_select(wl, scores)
    f64 = {n: oracle.bf16_bits_to_f64(bits[n]) for n in ("q", "k", "v")}
    oout, olse = oracle.block_sparse_attention(f64["q"], f64["k"], f64["v"], kept, wl.block, scale_of(wl))
    dref, dlref = oracle.dense_attention(f64["q"], f64["k"], f64["v"], scale_of(wl), block=wl.block)
    o = dict(qp=oqp, kp=okp, scores=scores, kept=kept, info=info, out=oout, lse=olse,
             dout=dref, dlse=dlref, f64=f64)
    res = (bits, dev, prob, sel, nb, g, o)
    _cache[wl.name] = res
    return res


@pytest.mark.parametrize("wl", CASES, ids=[c.name for c in CASES])
def test_pool(wl):
    _, _, _, _, _, g, o = run_case(wl)
    assert np.allclose(g["qp"], o["qp"], rtol=1e-6, atol=1e-7)
    assert np.allclose(g["kp"], o["kp"], rtol=1e-6, atol=1e-7)
    # the library rounds the float64 mean once: it must be the nearest float32
    assert np.array_equal(g["qp"], o["qp"].astype(np.float32))


@pytest.mark.parametrize("wl", CASES, ids=[c.name for c in CASES])
def test_select(wl):
    _, _, prob, sel, nb, g, o = run_case(wl)
    parity.check_idx_layout(g["idx"], g["cnt"], nb)
    rows_g = parity.gpu_rows(g["idx"], g["cnt"])
    rows_o = flat_rows(o["kept"])
    info = o["info"]
    n, same, problems = parity.compare_masks(rows_o, rows_g, o["scores"], info["mode"], k=info["k"],
                                             tau=info["tau"], forced=info["forced"])
    assert not problems, problems[:5]
    # the dense mask agrees with the index lists
    m = g["mask"].reshape(-1, nb)
    for r, row in enumerate(rows_g):
        assert m[r].sum() == len(row) and all(m[r, j] == 1 for j in row)
    if info["mode"] == "topk":
        assert np.all(g["cnt"] == info["k"])
    say(f"[select {wl.name}] rows={n} identical={same}")


@pytest.mark.parametrize("wl", CASES, ids=[c.name for c in CASES])
def test_sparse_attention_oracle_idx(wl):
    """The kernel fed the oracle's own index lists (no near-tie flips can leak)."""
    bits, dev, prob, sel, nb, g, o = run_case(wl)
    kmax = sva.max_keep(prob, sel)
    idx, cnt = oracle.kept_to_arrays(o["kept"], nb, kmax)
    out, lse = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], torch.from_numpy(idx).cuda(),
                                    torch.from_numpy(cnt).cuda(), want_lse=True)
    torch.cuda.synchronize()
    valid = np.ones(o["out"].shape, dtype=bool)
    mx, mean = parity.attention_errors(out.float().cpu().numpy(), o["out"], valid)
    assert mx <= parity.MAX_ABS and mean <= parity.MEAN_ABS, (mx, mean)
    assert np.max(np.abs(lse.cpu().numpy() - o["lse"])) <= parity.LSE_TOL


@pytest.mark.parametrize("wl", CASES, ids=[c.name for c in CASES])
def test_end_to_end(wl):
    """GPU pool -> GPU select -> GPU attention, checked on rows with identical masks."""
    _, _, prob, sel, nb, g, o = run_case(wl)
    rows_g = parity.gpu_rows(g["idx"], g["cnt"])
    rows_o = flat_rows(o["kept"])
    B, H, N, D = o["out"].shape
    valid = np.zeros((B, H, N, D), dtype=bool)
    r = 0
    for b in range(B):
        for h in range(H):
            for i in range(nb):
                if set(rows_g[r]) == set(rows_o[r]):
                    valid[b, h, i * wl.block:(i + 1) * wl.block] = True
                r += 1
    assert valid.any()
    mx, mean = parity.attention_errors(g["out"], o["out"], valid)
    assert mx <= parity.MAX_ABS and mean <= parity.MEAN_ABS, (mx, mean)
    say(f"[e2e {wl.name}] max={mx:.3e} mean={mean:.3e}")


@pytest.mark.parametrize("wl", CASES, ids=[c.name for c in CASES])
def test_dense(wl):
    _, _, _, _, _, g, o = run_case(wl)
    valid = np.ones(o["dout"].shape, dtype=bool)
    mx, mean = parity.attention_errors(g["dout"], o["dout"], valid)
    assert mx <= parity.MAX_ABS and mean <= parity.MEAN_ABS, (mx, mean)
    assert np.max(np.abs(g["dlse"] - o["dlse"])) <= parity.LSE_TOL


def _small(seed=7, D=128, S=64, grid=(3, 10, 13), B=1, H=2):
    wl = SC(f"adhoc_{seed}", B, H, D, grid, S, "topk", keep_ratio=0.5, seed=seed)
    bits = inputs.generate(wl)
    return wl, bits, device_inputs(bits), sva.problem_for(wl)


def test_degenerate_index_lists():
    """Empty rows -> zeros and -inf; out-of-range entries skipped; duplicates
    attended twice; order irrelevant; counts clamped to kmax."""
    wl, bits, dev, prob = _small(seed=11)
    nb = sva.num_blocks(prob)        # 7 blocks, last holds 6 tokens
    kmax = 5
    rows = [
        [],                      # empty
        [6, 0, 3],               # unsorted, includes the partial last block
        [-1, 2, nb, 9999, 4],    # out-of-range entries must be skipped
        [1, 1, 5],               # duplicate block
        [0, 1, 2, 3, 4],         # full row
        [5],
        [6],                     # only the partial block
    ]
    idx = np.full((1, 2, nb, kmax), -1, dtype=np.int32)
    cnt = np.zeros((1, 2, nb), dtype=np.int32)
    for h in range(2):
        for i, row in enumerate(rows):
            idx[0, h, i, :len(row)] = row
            cnt[0, h, i] = len(row)
    cnt[0, 1, 4] = 99            # count above kmax is clamped to kmax
    out, lse = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], torch.from_numpy(idx).cuda(),
                                    torch.from_numpy(cnt).cuda(), want_lse=True)
    torch.cuda.synchronize()
    out = out.float().cpu().numpy()
    lse = lse.cpu().numpy()
    expect = [[[j for j in row if 0 <= j < nb] for row in rows] for _ in range(2)]
    f64 = {n: oracle.bf16_bits_to_f64(bits[n]) for n in ("q", "k", "v")}
    ref, rlse = oracle.block_sparse_attention(f64["q"], f64["k"], f64["v"], [expect], wl.block, scale_of(wl))
    assert np.all(out[0, :, :64] == 0) and np.all(np.isneginf(lse[0, :, :64]))
    valid = np.ones(ref.shape, dtype=bool)
    valid[0, :, :64] = False
    mx, mean = parity.attention_errors(out, ref, valid)
    assert mx <= parity.MAX_ABS and mean <= parity.MEAN_ABS, (mx, mean)
    fin = np.isfinite(rlse)
    assert np.max(np.abs(lse[fin] - rlse[fin])) <= parity.LSE_TOL


def test_constant_values_and_fp32_output():
    wl, bits, dev, prob = _small(seed=12, D=112, S=128, grid=(2, 9, 14))
    ones = torch.ones_like(dev["v"])
    prob32 = sva.problem_for(wl, out_dtype="f32")
    out, _ = sva.dense_attention(prob32, dev["q"], dev["k"], ones)
    torch.cuda.synchronize()
    assert out.dtype == torch.float32
    assert torch.max(torch.abs(out - 1.0)).item() <= 4e-3
    # fp32 output is held to a tighter mean error than bf16 output
    f64 = {n: oracle.bf16_bits_to_f64(bits[n]) for n in ("q", "k", "v")}
    ref, _ = oracle.dense_attention(f64["q"], f64["k"], f64["v"], scale_of(wl), block=wl.block)
    o32, _ = sva.dense_attention(prob32, dev["q"], dev["k"], dev["v"])
    torch.cuda.synchronize()
    mx, mean = parity.attention_errors(o32.cpu().numpy(), ref, np.ones(ref.shape, dtype=bool))
    assert mx <= 1e-2 and mean <= 1e-3, (mx, mean)


@pytest.mark.parametrize("S", [128, 64])
def test_keep_all_equals_dense_and_determinism(S):
    """Keep-all lists against dense attention, bit for bit (at S = 64 dense
    attention runs as 128-token query tiles: the same keys in the same chunks
    and order), and repeat runs bit for bit."""
    wl, bits, dev, prob = _small(seed=13, D=128, S=S, grid=(3, 10, 13))
    nb = sva.num_blocks(prob)
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    idx, cnt, _ = sva.select_blocks(prob, sva.select_topk(1.0), qp, kp)
    torch.cuda.synchronize()
    assert np.all(cnt.cpu().numpy() == nb)
    assert np.array_equal(idx.cpu().numpy()[0, 0, 0], np.arange(nb))
    o1, l1 = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], idx, cnt, want_lse=True)
    o2, l2 = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], idx, cnt, want_lse=True)
    od, ld = sva.dense_attention(prob, dev["q"], dev["k"], dev["v"], want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)      # bitwise repeatable
    assert torch.equal(o1, od) and torch.equal(l1, ld)      # same block order as dense


def test_block_pairs_match_single_blocks():
    """At block 64 and D = 128, rows of at least 15% of the blocks (kmax) run
    as pairs of neighbouring query blocks over the union of their lists;
    shorter rows one block at a time.  The same lists in longer rows (padded with -1 past the
    counts) take the pair path: outputs and LSE must match bit for bit, with an
    odd block count (the last pair has one block)."""
    wl, bits, dev, prob = _small(seed=16, D=128, S=64, grid=(3, 10, 13), H=2)
    nb = sva.num_blocks(prob)
    assert nb % 2 == 1
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    idx, cnt, _ = sva.select_blocks(prob, sva.select_topk(topk=1), qp, kp)
    assert idx.shape[-1] * 20 < 3 * nb                      # single-block path
    wide = torch.full((1, 2, nb, nb), -1, dtype=torch.int32, device="cuda")
    wide[..., :idx.shape[-1]] = idx
    o1, l1 = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], idx, cnt, want_lse=True)
    o2, l2 = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], wide, cnt, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_segment_order_covers_every_row():
    """Sparse lists at S=128 hand rows to the XCDs in segments of 8 x 128; with
    3 heads of 393 blocks (ragged last block) there are 1179 rows: one whole
    segment and a 155-row tail.  Keep-all lists must reproduce dense attention
    bit for bit on every row, written over a NaN-filled output."""
    wl, bits, dev, prob = _small(seed=15, D=128, S=128, grid=(8, 40, 157), H=3)
    nb = sva.num_blocks(prob)
    assert nb == 393 and 3 * nb > 8 * 128
    idx = torch.arange(nb, dtype=torch.int32, device="cuda").expand(1, 3, nb, nb).contiguous()
    cnt = torch.full((1, 3, nb), nb, dtype=torch.int32, device="cuda")
    out = torch.full_like(dev["q"], float("nan"))
    lse = torch.full((1, 3, wl.seq_len), float("nan"), device="cuda")
    sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], idx, cnt, out=out, want_lse=True, lse=lse)
    od, ld = sva.dense_attention(prob, dev["q"], dev["k"], dev["v"], want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(out, od) and torch.equal(lse, ld)


def test_custom_scale():
    wl, bits, dev, prob = _small(seed=14, D=64, S=64, grid=(2, 8, 9))
    c = 0.3
    p = sva.problem_for(wl, softmax_scale=c)
    out, lse = sva.dense_attention(p, dev["q"], dev["k"], dev["v"], want_lse=True)
    torch.cuda.synchronize()
    f64 = {n: oracle.bf16_bits_to_f64(bits[n]) for n in ("q", "k", "v")}
    ref, rl = oracle.dense_attention(f64["q"], f64["k"], f64["v"], c, block=64)
    mx, mean = parity.attention_errors(out.float().cpu().numpy(), ref, np.ones(ref.shape, dtype=bool))
    assert mx <= parity.MAX_ABS and mean <= parity.MEAN_ABS
    assert np.max(np.abs(lse.cpu().numpy() - rl)) <= parity.LSE_TOL


def test_select_ties_go_to_lower_index():
    """Pooled summaries with exact ties: the lower block index must win, on the
    GPU exactly as in the oracle (the GPU scores the same float32 summaries)."""
    B, H, nb, D = 1, 1, 16, 64
    prob = sva.problem(B, H, nb * 64, D, (1, 1, nb * 64), 64)
    rng = np.random.default_rng(3)
    kp = rng.standard_normal((nb, D)).astype(np.float32)
    kp[9] = kp[3]
    kp[12] = kp[3]               # blocks 3, 9, 12 identical
    kp[5] = kp[7]
    qp = rng.standard_normal((nb, D)).astype(np.float32)
    qp[2] = kp[3]                # row 2 scores 3/9/12 highest, tied
    qt = torch.from_numpy(qp[None, None]).cuda()
    kt = torch.from_numpy(kp[None, None]).cuda()
    for k in (1, 2, 3, 5):
        idx, cnt, _ = sva.select_blocks(prob, sva.select_topk(0.0, k), qt, kt)
        torch.cuda.synchronize()
        s = oracle.block_scores(qp.astype(np.float64)[None, None], kp.astype(np.float64)[None, None],
                                1.0 / math.sqrt(D))
        want = oracle.select_topk(s, k)[0][0]
        assert parity.gpu_rows(idx.cpu().numpy(), cnt.cpu().numpy()) == want, k
        assert want[2][:1] == [3]        # of the tied 3/9/12 the lowest index comes first


@pytest.mark.parametrize("S,D", [(128, 128), (64, 128), (128, 112)])
def test_gradual_logit_growth_is_exact(S, D):
    """Logits rise by ~40 (log2 units) from one kept block to the next, so the
    row sum relative to the first chunk's maximum passes 2^64 after a few
    blocks and would reach ~2^127 by the last: the kernel must move its
    reference between blocks and still match the oracle."""
    B, H = 1, 1
    nblk = 5
    grid = (1, nblk * S // 16, 16)
    wl = SC(f"growth_{S}_{D}", B, H, D, grid, S, "topk", topk=nblk, seed=37)
    bits = inputs.generate(wl)
    f = {n: inputs.bf16_bits_to_f32(bits[n]).copy() for n in ("q", "k", "v")}
    c = scale_of(wl)
    f["q"][0, 0] = 1.0
    # key block b: every element equal, logits q.k * c = 40*b / log2(e)
    for b in range(nblk):
        val = 40.0 * b / (math.log2(math.e) * c * D) + 0.01
        f["k"][0, 0, b * S:(b + 1) * S] = val + 0.02 * f["k"][0, 0, b * S:(b + 1) * S]
    new_bits = {n: inputs._round_bf16(f[n]) for n in f}
    dev = device_inputs(new_bits)
    prob = sva.problem_for(wl)
    rows = [list(range(nblk)) for _ in range(nblk)]
    idx = np.array(rows, dtype=np.int32).reshape(1, 1, nblk, nblk)
    cnt = np.full((1, 1, nblk), nblk, dtype=np.int32)
    out, lse = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], torch.from_numpy(idx).cuda(),
                                    torch.from_numpy(cnt).cuda(), want_lse=True)
    dout, dlse = sva.dense_attention(prob, dev["q"], dev["k"], dev["v"], want_lse=True)
    torch.cuda.synchronize()
    f64 = {n: oracle.bf16_bits_to_f64(new_bits[n]) for n in ("q", "k", "v")}
    ref, rlse = oracle.block_sparse_attention(f64["q"], f64["k"], f64["v"], [[rows]], S, c)
    assert rlse.max() > 100.0                      # the regime this test is about
    for o_, l_ in ((out, lse), (dout, dlse)):
        o = o_.float().cpu().numpy()
        assert np.isfinite(o).all()
        mx, mean = parity.attention_errors(o, ref, np.ones(ref.shape, dtype=bool))
        assert mx <= parity.MAX_ABS and mean <= parity.MEAN_ABS, (mx, mean)
        err = np.abs(l_.cpu().numpy() - rlse)
        assert np.all(err <= parity.LSE_TOL + 1e-5 * np.abs(rlse)), err.max()


def test_block_pair_overflow_is_recomputed():
    """The block-64 pair kernel (D = 128) with a later kept block whose logits
    exceed the first chunk's reference by about 1000 (log2 units): the pair
    is marked and recomputed with per-iteration rescaling, and every query
    block matches the oracle."""
    S, D = 64, 128
    wl = SC("overflow_pairs", 1, 1, D, (4, 8, 16), S, "topk", topk=2, seed=33)   # N = 512, 8 blocks
    bits = inputs.generate(wl)
    f = {n: inputs.bf16_bits_to_f32(bits[n]).copy() for n in ("q", "k", "v")}
    f["k"][0, 0, 0:64] *= 1e-3
    f["q"][0, 0, 128:256] = 8.0                      # query blocks 2 and 3
    f["k"][0, 0, 384:512] = 8.0                      # key blocks 6 and 7
    new_bits = {n: inputs._round_bf16(f[n]) for n in f}
    dev = device_inputs(new_bits)
    prob = sva.problem_for(wl)
    rows = [[0, 1], [1, 2], [0, 6], [0, 7], [3, 4], [4, 5], [5, 6], [6, 7]]
    idx = np.array(rows, dtype=np.int32).reshape(1, 1, 8, 2)
    cnt = np.full((1, 1, 8), 2, dtype=np.int32)
    assert 2 * 20 >= 3 * 8                          # the pair path
    out, lse = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], torch.from_numpy(idx).cuda(),
                                    torch.from_numpy(cnt).cuda(), want_lse=True)
    torch.cuda.synchronize()
    f64 = {n: oracle.bf16_bits_to_f64(new_bits[n]) for n in ("q", "k", "v")}
    ref, rlse = oracle.block_sparse_attention(f64["q"], f64["k"], f64["v"], [[rows]], S, scale_of(wl))
    assert rlse.max() > 400.0                        # the regime this test is about
    o = out.float().cpu().numpy()
    assert np.isfinite(o).all()
    mx, mean = parity.attention_errors(o, ref, np.ones(ref.shape, dtype=bool))
    assert mx <= parity.MAX_ABS and mean <= parity.MEAN_ABS, (mx, mean)
    err = np.abs(lse.cpu().numpy() - rlse)
    assert np.all(err <= parity.LSE_TOL + 1e-5 * np.abs(rlse)), err.max()


@pytest.mark.parametrize("S,D", [(128, 128), (128, 112), (128, 64)])
def test_logit_growth_beyond_fixed_reference_is_exact(S, D):
    """Block-size-128 kernels fix the softmax reference max from the first key
    chunk.  Here a later kept block's logits exceed it by about 1000 (log2
    units), which overflows that reference; the block must be recomputed with
    per-iteration rescaling and still match the oracle, while other query
    blocks keep their normal results."""
    B, H, grid = 1, 1, (4, 8, 16)           # N = 512, 4 blocks of 128
    wl = SC(f"overflow_{S}_{D}", B, H, D, grid, S, "topk", topk=2, seed=31)
    bits = inputs.generate(wl)
    N = wl.seq_len
    # block 0 keys ~0 (logits ~0 for every query), block 3 keys large and aligned with queries 128..255
    f = {n: inputs.bf16_bits_to_f32(bits[n]).copy() for n in ("q", "k", "v")}
    f["k"][0, 0, 0:128] *= 1e-3
    f["q"][0, 0, 128:256] = 8.0
    f["k"][0, 0, 384:512] = 8.0
    new_bits = {n: inputs._round_bf16(f[n]) for n in f}
    dev = device_inputs(new_bits)
    prob = sva.problem_for(wl)
    rows = [[0, 1], [0, 3], [1, 2], [2, 3]]          # query block 1: first block 0, then the huge block 3
    idx = np.array(rows, dtype=np.int32).reshape(1, 1, 4, 2)
    cnt = np.full((1, 1, 4), 2, dtype=np.int32)
    out, lse = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], torch.from_numpy(idx).cuda(),
                                    torch.from_numpy(cnt).cuda(), want_lse=True)
    torch.cuda.synchronize()
    f64 = {n: oracle.bf16_bits_to_f64(new_bits[n]) for n in ("q", "k", "v")}
    ref, rlse = oracle.block_sparse_attention(f64["q"], f64["k"], f64["v"], [[rows]], S, scale_of(wl))
    o = out.float().cpu().numpy()
    assert np.isfinite(o).all()
    mx, mean = parity.attention_errors(o, ref, np.ones(ref.shape, dtype=bool))
    assert mx <= parity.MAX_ABS and mean <= parity.MEAN_ABS, (mx, mean)
    # absolute bf16-probability bound plus float32 relative error of a ~700 LSE
    err = np.abs(lse.cpu().numpy() - rlse)
    assert np.all(err <= parity.LSE_TOL + 1e-5 * np.abs(rlse)), err.max()
