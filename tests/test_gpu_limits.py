"""GPU parity at the size limits of the boundary: 2048 key blocks per row (the
most the selection kernel holds in registers) in both selection modes (and
every kernel shape the selection launch picks on the way there), with
attention on sampled query blocks in bf16 and fp8, fp8 dense attention at
2047 blocks (the longest kept-block list the fp8 kernel holds in LDS), and
4096 blocks for the block-pair kernel and the first-order remainder."""
import numpy as np
import pytest

import oracle
import oracle.fp8_attention as of8
import oracle.remainder as orem
import paper_2606_23743_amd as sva
from paper_2606_23743_amd import inputs, workloads

from . import parity
from .gpu_cases import device_inputs, flat_rows, oracle_select, say, scale_of
from .test_gpu_fp8 import _check_attention, _dequantised

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SC = workloads.small_case
LIMIT_CASES = [
    SC("nb2048_topk", 1, 1, 64, (2, 256, 256), 64, "topk", keep_ratio=0.05, seed=211),
    SC("nb2048_mass", 1, 1, 64, (2, 256, 256), 64, "mass", mass_threshold=0.9, max_keep_ratio=0.3,
       force_first_frame=False, seed=212),
]


SELECT_CASES = [
    SC("d112_nb1536_topk", 1, 2, 112, (6, 64, 256), 64, "topk", keep_ratio=0.1, seed=213),
    SC("d112_nb1536_mass", 1, 2, 112, (6, 64, 256), 64, "mass", mass_threshold=0.9, max_keep_ratio=0.3,
       force_first_frame=True, seed=214),
]


# one case per kernel shape the selection launch picks between 9 and 20
# chunks of 64 blocks (12, 14, 16 and 20 registers of scores per lane; eight
# waves of two rows or sixteen of one; the 20-chunk top-k shape with its
# registers capped), in both rules
SHAPE_CASES = [
    SC("nb700_topk", 1, 2, 64, (5, 80, 112), 64, "topk", keep_ratio=0.2, seed=215),
    SC("nb870_topk", 1, 2, 128, (5, 96, 116), 64, "topk", keep_ratio=0.15, seed=216),
    SC("nb1000_topk", 1, 2, 64, (5, 80, 160), 64, "topk", keep_ratio=0.2, seed=221),
    SC("nb1100_topk", 1, 2, 64, (5, 80, 176), 64, "topk", keep_ratio=0.25, seed=217),
    SC("nb1280_topk", 1, 1, 128, (5, 64, 256), 64, "topk", keep_ratio=0.1, seed=218),
    SC("nb1100_mass", 1, 2, 64, (5, 80, 176), 64, "mass", mass_threshold=0.9, max_keep_ratio=0.3,
       force_first_frame=True, seed=219),
    SC("nb1280_mass", 1, 1, 128, (5, 64, 256), 64, "mass", mass_threshold=0.8, max_keep_ratio=0.2,
       force_first_frame=False, seed=220),
]


@pytest.mark.parametrize("wl", SELECT_CASES, ids=[c.name for c in SELECT_CASES])
def test_selection_head_dim_112_past_1024_blocks(wl):
    """Selection with D = 112 (score steps of 28 channels per lane group) at
    1536 blocks per row, where a lane holds 24 registers of scores: every
    row's kept list against the oracle's."""
    _selection_every_row(wl, 1536)


@pytest.mark.parametrize("wl", SHAPE_CASES, ids=[c.name for c in SHAPE_CASES])
def test_selection_kernel_shapes(wl):
    """Every row's kept list against the oracle's at block counts that select
    each of the selection kernel's shapes from 9 to 20 chunks."""
    _selection_every_row(wl, wl.seq_len // wl.block)


def _selection_every_row(wl, nb_expected):
    say(f"[limits {wl.name}] N={wl.seq_len} nB={wl.seq_len // wl.block}")
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    sel = sva.select_for(wl)
    nb = sva.num_blocks(prob)
    assert nb == nb_expected
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    idx, cnt, mask = sva.select_blocks(prob, sel, qp, kp, want_mask=True)
    torch.cuda.synchronize()
    f64 = {n: oracle.bf16_bits_to_f64(bits[n]) for n in ("q", "k")}
    scores = oracle.block_scores(oracle.pool_blocks(f64["q"], wl.block), oracle.pool_blocks(f64["k"], wl.block),
                                 scale_of(wl))
    kept, info = oracle_select(wl, scores)
    idx_np, cnt_np = idx.cpu().numpy(), cnt.cpu().numpy()
    parity.check_idx_layout(idx_np, cnt_np, nb)
    # the optional mask says exactly what the lists say
    m_np = mask.cpu().numpy().reshape(-1, nb)
    want = np.zeros_like(m_np)
    for r, (row, c) in enumerate(zip(idx_np.reshape(-1, idx_np.shape[-1]), cnt_np.reshape(-1))):
        want[r, row[:c]] = 1
    assert np.array_equal(m_np, want)
    n, same, problems = parity.compare_masks(flat_rows(kept), parity.gpu_rows(idx_np, cnt_np), scores,
                                             info["mode"], k=info["k"], tau=info["tau"], forced=info["forced"])
    assert not problems, problems[:5]
    say(f"[limits {wl.name}] selection rows={n} identical={same}")


def _kept_arrays(kept, nb):
    kmax = max(1, max(len(r) for b in kept for h in b for r in h))
    idx, cnt = oracle.kept_to_arrays(kept, nb, kmax)
    return (torch.from_numpy(np.ascontiguousarray(idx, dtype=np.int32)).cuda(),
            torch.from_numpy(np.ascontiguousarray(cnt, dtype=np.int32)).cuda())


@pytest.mark.parametrize("wl", LIMIT_CASES, ids=[c.name for c in LIMIT_CASES])
def test_selection_and_attention_at_2048_blocks(wl):
    say(f"[limits {wl.name}] N={wl.seq_len} nB={wl.seq_len // wl.block}")
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    sel = sva.select_for(wl)
    nb = sva.num_blocks(prob)
    assert nb == 2048
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    idx, cnt, _ = sva.select_blocks(prob, sel, qp, kp)
    torch.cuda.synchronize()
    f64 = {n: oracle.bf16_bits_to_f64(bits[n]) for n in ("q", "k", "v")}
    oqp = oracle.pool_blocks(f64["q"], wl.block)
    okp = oracle.pool_blocks(f64["k"], wl.block)
    scores = oracle.block_scores(oqp, okp, scale_of(wl))
    kept, info = oracle_select(wl, scores)
    idx_np, cnt_np = idx.cpu().numpy(), cnt.cpu().numpy()
    parity.check_idx_layout(idx_np, cnt_np, nb)
    n, same, problems = parity.compare_masks(flat_rows(kept), parity.gpu_rows(idx_np, cnt_np), scores,
                                             info["mode"], k=info["k"], tau=info["tau"], forced=info["forced"])
    assert not problems, problems[:5]
    say(f"[limits {wl.name}] selection rows={n} identical={same}")

    # attention on sampled query blocks with the oracle's lists, bf16 and fp8
    oidx, ocnt = _kept_arrays(kept, nb)
    out, lse = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], oidx, ocnt, want_lse=True)
    quant = sva.quantize_fp8(prob, dev["q"], dev["k"], dev["v"])
    out8, lse8 = sva.sparse_attention_fp8(prob, quant, oidx, ocnt, want_lse=True)
    torch.cuda.synchronize()
    rows = [0, 1, 777, 1500, nb - 1]
    ref, rlse = oracle.block_sparse_attention(f64["q"], f64["k"], f64["v"], kept, wl.block, scale_of(wl),
                                              rows=[(0, 0, i) for i in rows])
    o = out.float().cpu().numpy()
    for i in rows:
        sl = slice(i * wl.block, (i + 1) * wl.block)
        mx, mean = parity.attention_errors(o[0, 0, sl], ref[0, 0, sl], np.ones(ref[0, 0, sl].shape, dtype=bool))
        assert mx <= parity.MAX_ABS and mean <= parity.MEAN_ABS, (i, mx, mean)
        assert np.all(np.abs(lse.cpu().numpy()[0, 0, sl] - rlse[0, 0, sl]) <= parity.LSE_TOL), i
    qref = _dequantised(bits, wl.block, 0, 0)
    rms, pred = _check_attention(out8.float().cpu().numpy().astype(np.float64)[0, 0], lse8.cpu().numpy()[0, 0],
                                 qref, kept[0][0], wl.block, of8.LN2, rows)
    assert rms <= 2.0 * pred + 5e-4, (rms, pred)
    say(f"[limits {wl.name}] fp8 rms {rms:.2e} (model {pred:.2e})")


def test_block_pairs_at_4096_blocks():
    """The block-pair kernel at its largest size: D = 128, 64-token blocks,
    nB = 4096 (128 bitmap words, two compaction steps), rows of 16% of the
    blocks from the oracle's selection (the selection kernel itself takes at
    most 2048 blocks per row and says so); attention on sampled rows (first
    and last pairs included) against the oracle."""
    wl = SC("nb4096_pairs", 1, 1, 128, (4, 256, 256), 64, "topk", keep_ratio=0.16, seed=214)
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    nb = sva.num_blocks(prob)
    assert nb == 4096
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    with pytest.raises(sva.SvaError) as err:
        sva.select_blocks(prob, sva.select_for(wl), qp, kp)
    assert err.value.status == 4                            # unsupported block count
    f64 = {n: oracle.bf16_bits_to_f64(bits[n]) for n in ("q", "k", "v")}
    scores = oracle.block_scores(oracle.pool_blocks(f64["q"], wl.block), oracle.pool_blocks(f64["k"], wl.block),
                                 scale_of(wl))
    kept, _ = oracle_select(wl, scores)
    oidx, ocnt = _kept_arrays(kept, nb)
    assert oidx.shape[-1] * 20 >= 3 * nb                    # the pair path
    out, lse = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], oidx, ocnt, want_lse=True)
    torch.cuda.synchronize()
    rows = [0, 1, 2047, 4094, 4095]
    ref, rlse = oracle.block_sparse_attention(f64["q"], f64["k"], f64["v"], kept, wl.block, scale_of(wl),
                                              rows=[(0, 0, i) for i in rows])
    o = out.float().cpu().numpy()
    for i in rows:
        sl = slice(i * wl.block, (i + 1) * wl.block)
        mx, mean = parity.attention_errors(o[0, 0, sl], ref[0, 0, sl], np.ones(ref[0, 0, sl].shape, dtype=bool))
        assert mx <= parity.MAX_ABS and mean <= parity.MEAN_ABS, (i, mx, mean)
        assert np.all(np.abs(lse.cpu().numpy()[0, 0, sl] - rlse[0, 0, sl]) <= parity.LSE_TOL), i
    say(f"[limits nb4096 pairs] rows {rows} within the parity bounds")


def test_remainder_at_4096_blocks():
    """The first-order remainder at its largest block count, nB = 4096 (128
    bitmap words per row, no padding rows, 4096-row weight chunks), on the
    oracle's lists, sampled rows (first and last included) against the
    oracle with the remainder's bounds."""
    wl = SC("nb4096_remainder", 1, 1, 128, (4, 256, 256), 64, "topk", keep_ratio=0.05, seed=215)
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    nb = sva.num_blocks(prob)
    assert nb == 4096
    f64 = {n: oracle.bf16_bits_to_f64(bits[n]) for n in ("q", "k", "v")}
    scores = oracle.block_scores(oracle.pool_blocks(f64["q"], wl.block), oracle.pool_blocks(f64["k"], wl.block),
                                 scale_of(wl))
    kept, _ = oracle_select(wl, scores)
    oidx, ocnt = _kept_arrays(kept, nb)
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    out, lse = sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, oidx, ocnt, want_lse=True)
    torch.cuda.synchronize()
    rows = [0, 1, 2047, 4094, 4095]
    c = scale_of(wl)
    ref, rlse = orem.remainder_attention(f64["q"], f64["k"], f64["v"], kept, wl.block, c,
                                         rows=[(0, 0, i) for i in rows], weight=parity.KERNEL_REMAINDER_FORM)
    ref0, _ = orem.remainder_attention(f64["q"], f64["k"], f64["v"], kept, wl.block, c,
                                       rows=[(0, 0, i) for i in rows], first_order=False,
                                       weight=parity.KERNEL_REMAINDER_FORM)
    o = out.float().cpu().numpy()
    kbar = oracle.pool_blocks(f64["k"][0, 0], wl.block)
    for i in rows:
        sl = slice(i * wl.block, (i + 1) * wl.block)
        excess, mean, mean_bound = parity.remainder_errors(o[0, 0, sl], ref[0, 0, sl], ref[0, 0, sl] - ref0[0, 0, sl],
                                                           True)
        assert excess <= 0.0 and mean <= mean_bound, (i, excess, mean, mean_bound)
        bound = parity.remainder_lse_bound(f64["q"][0, 0, sl], kbar, c)
        assert np.all(np.abs(lse.cpu().numpy()[0, 0, sl] - rlse[0, 0, sl]) <= bound), i
    say(f"[limits nb4096 remainder] rows {rows} within the remainder bounds")


def test_fp8_dense_at_2047_blocks():
    wl = SC("nb2047_dense", 1, 1, 64, (23, 89, 64), 64, "topk", topk=1, seed=213)
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    assert sva.num_blocks(prob) == 2047
    quant = sva.quantize_fp8(prob, dev["q"], dev["k"], dev["v"])
    out8, lse8 = sva.dense_attention_fp8(prob, quant, want_lse=True)
    torch.cuda.synchronize()
    qref = _dequantised(bits, wl.block, 0, 0)
    rows = [0, 1023, 2046]
    every = [list(range(2047))] * 2047
    rms, pred = _check_attention(out8.float().cpu().numpy().astype(np.float64)[0, 0], lse8.cpu().numpy()[0, 0],
                                 qref, every, wl.block, of8.LN2, rows)
    assert rms <= 2.0 * pred + 5e-4, (rms, pred)
    say(f"[limits dense fp8 nB=2047] rms {rms:.2e} (model {pred:.2e})")
