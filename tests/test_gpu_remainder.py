"""GPU parity of the first-order remainder of dropped blocks (the block
moments, and attention over the kept blocks plus the remainder) against the
oracle on reduced shapes: every head dim and block size, ragged tails, a row
count that is not a multiple of the 32-block chunks, the block-pair path of
the kept part, and degenerate lists (empty rows, every block kept, out-of-range
entries, duplicates).  The index lists come from the oracle's own selection;
the pooled means the GPU call takes come from the GPU's pooling step.
"""
import numpy as np
import pytest

import oracle
import oracle.remainder as orem
import paper_2606_23743_amd as sva
from paper_2606_23743_amd import inputs, workloads

from . import parity
from .gpu_cases import device_inputs, oracle_pool_all, oracle_select, say, scale_of

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SC = workloads.small_case
CASES = [
    SC("rem_d128_s128", 1, 2, 128, (4, 10, 13), 128, "topk", keep_ratio=0.2, seed=301),
    SC("rem_d128_s64_pairs", 1, 2, 128, (5, 8, 9), 64, "topk", keep_ratio=0.3, seed=302),
    SC("rem_d112_s64", 2, 1, 112, (3, 10, 13), 64, "topk", keep_ratio=0.1, seed=303),
    SC("rem_d64_s128", 1, 3, 64, (4, 10, 13), 128, "topk", topk=2, seed=304),
    SC("rem_d112_s128_mass", 1, 2, 112, (6, 9, 11), 128, "mass", mass_threshold=0.8,
       max_keep_ratio=0.4, force_first_frame=True, seed=305),
    SC("rem_d64_s64_40blocks", 1, 2, 64, (5, 16, 32), 64, "topk", keep_ratio=0.1, seed=306),
    SC("rem_d128_s64_one_block", 1, 2, 128, (1, 5, 7), 64, "topk", topk=1, seed=307),
]


def _degenerate(kept, nb, rng):
    """Rows 0..3 of every head replaced by: empty, every block, out-of-range
    and repeated entries, one block listed twice."""
    for b in kept:
        for h in b:
            h[0] = []
            if nb > 1:
                h[1] = list(range(nb))
            if nb > 2:
                h[2] = [-3, nb, int(rng.integers(nb)), nb + 7]
            if nb > 3:
                j = int(rng.integers(nb))
                h[3] = [j, j]
    return kept


def _arrays(kept, nb):
    kmax = max(1, max(len(r) for b in kept for h in b for r in h))
    idx = np.full((len(kept), len(kept[0]), nb, kmax), -1, dtype=np.int32)
    cnt = np.zeros((len(kept), len(kept[0]), nb), dtype=np.int32)
    for bi, b in enumerate(kept):
        for hi, h in enumerate(b):
            for i, row in enumerate(h):
                idx[bi, hi, i, :len(row)] = row
                cnt[bi, hi, i] = len(row)
    return torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda()


def _oracle_lists(wl, bits):
    """The oracle's own selection, as nested [B][H][nB] lists of ints."""
    oqp, okp = oracle_pool_all(bits, wl.block)
    kept, _ = oracle_select(wl, oracle.block_scores(oqp, okp, scale_of(wl)))
    return [[[list(map(int, r)) for r in h] for h in b] for b in kept]


@pytest.mark.parametrize("wl", CASES, ids=[c.name for c in CASES])
def test_block_moments(wl):
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    say(f"[remainder moments {wl.name}] N={wl.seq_len} D={wl.head_dim} S={wl.block}")
    kbar, vbar, mom = sva.block_moments(prob, dev["k"], dev["v"])
    torch.cuda.synchronize()
    gk, gv, gm = (t.float().cpu().numpy().astype(np.float64) for t in (kbar, vbar, mom))
    for b in range(wl.batch):
        for h in range(wl.heads):
            k = oracle.bf16_bits_to_f64(bits["k"][b, h])
            v = oracle.bf16_bits_to_f64(bits["v"][b, h])
            okb, ovb, om = orem.block_moments(k, v, wl.block)
            # means: float32 sums rounded once to bf16
            assert np.all(np.abs(gk[b, h] - okb) <= 2.0 ** -8 * np.abs(okb) + 1e-6)
            assert np.all(np.abs(gv[b, h] - ovb) <= 2.0 ** -8 * np.abs(ovb) + 1e-6)
            # moments: float32 sums of exact products less the outer product of the
            # sums (bounded as if K - kbar were rounded to bf16), one bf16 rounding
            bound = np.empty_like(om)
            for j, (a, e) in enumerate(oracle.block_bounds(wl.seq_len, wl.block)):
                dk = np.abs(k[a:e] - okb[j])
                bound[j] = 2.0 ** -7 * (np.abs(v[a:e]).T @ dk) + 2.0 ** -8 * np.abs(om[j]) + 1e-5
            err = np.abs(gm[b, h] - om)
            assert np.all(err <= bound), (float(err.max()), float((err - bound).max()))


@pytest.mark.parametrize("wl", CASES, ids=[c.name for c in CASES])
@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_remainder_attention(wl, out_dtype):
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl, out_dtype=out_dtype)
    nb = sva.num_blocks(prob)
    say(f"[remainder {wl.name} {out_dtype}] N={wl.seq_len} nB={nb} D={wl.head_dim} S={wl.block}")
    kept = _oracle_lists(wl, bits)
    kept = _degenerate(kept, nb, np.random.default_rng(wl.seed))
    idx, cnt = _arrays(kept, nb)
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    out, lse = sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt, want_lse=True)
    out2, lse2 = sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt,
                                                want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(out, out2) and torch.equal(lse, lse2), "remainder attention is not deterministic"
    got = out.float().cpu().numpy()
    glse = lse.cpu().numpy()
    c = scale_of(wl)
    worst = 0.0
    for b in range(wl.batch):
        for h in range(wl.heads):
            f = {n: oracle.bf16_bits_to_f64(bits[n][b, h])[None, None] for n in ("q", "k", "v")}
            ref, rlse = orem.remainder_attention(f["q"], f["k"], f["v"], [[kept[b][h]]], wl.block, c,
                                                 weight=parity.KERNEL_REMAINDER_FORM)
            ref0, _ = orem.remainder_attention(f["q"], f["k"], f["v"], [[kept[b][h]]], wl.block, c,
                                               first_order=False, weight=parity.KERNEL_REMAINDER_FORM)
            excess, mean, mean_bound = parity.remainder_errors(got[b, h], ref[0, 0], ref[0, 0] - ref0[0, 0],
                                                               out_dtype == "bf16")
            assert excess <= 0.0 and mean <= mean_bound, ((b, h), excess, mean, mean_bound)
            # against the plain expansion (the query's own first-order weight):
            # the same bounds widened by the exact gap between the two forms
            plain, plse = orem.remainder_attention(f["q"], f["k"], f["v"], [[kept[b][h]]], wl.block, c,
                                                   weight="query")
            excess_p, gap_mean, gap_max = parity.remainder_errors_vs_plain(got[b, h], plain[0, 0], ref[0, 0],
                                                                           ref[0, 0] - ref0[0, 0],
                                                                           out_dtype == "bf16")
            assert excess_p <= 0.0, ((b, h), excess_p)
            assert np.abs(plse - rlse).max() < 1e-9          # the two forms share the denominator
            if b == 0 and h == 0:
                say(f"[remainder {wl.name} {out_dtype}] block-mean vs plain expansion: mean |gap| "
                    f"{gap_mean:.2e}, max {gap_max:.2e}")
            lse_bound = parity.remainder_lse_bound(f["q"][0, 0], oracle.pool_blocks(f["k"][0, 0], wl.block), c)
            assert np.all(np.abs(glse[b, h] - rlse[0, 0]) <= lse_bound), (b, h)
            worst = max(worst, float(np.max(np.abs(got[b, h] - ref[0, 0]))))
    say(f"[remainder {wl.name} {out_dtype}] max |err| {worst:.2e}")


def test_keep_all_equals_the_sparse_result():
    """Every block kept: nothing is dropped, so the result is the kept-block
    attention, merged through a float32 buffer (within one bf16 step)."""
    wl = SC("rem_keep_all", 1, 2, 128, (4, 10, 13), 64, "topk", keep_ratio=1.0, seed=308)
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    nb = sva.num_blocks(prob)
    every = [[[list(range(nb)) for _ in range(nb)] for _ in range(wl.heads)]]
    idx, cnt = _arrays(every, nb)
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    rem, rlse = sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt, want_lse=True)
    sp, slse = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], idx, cnt, want_lse=True)
    torch.cuda.synchronize()
    a, b = rem.float().cpu().numpy(), sp.float().cpu().numpy()
    step = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(b), 2.0 ** -126))) - 7)
    assert np.all(np.abs(a - b) <= step)
    assert np.mean(a == b) > 0.99
    assert np.allclose(rlse.cpu().numpy(), slse.cpu().numpy(), rtol=1e-6, atol=1e-6)


def test_workspace_is_reusable_and_sized_by_the_call():
    """One workspace serves two calls of different sizes; the second, smaller
    call sees the first call's leftovers and must not depend on them."""
    wl1 = CASES[0]
    wl2 = SC("rem_small_after_large", 1, 1, 128, (2, 6, 7), 128, "topk", keep_ratio=0.3, seed=309)
    p1, p2 = sva.problem_for(wl1), sva.problem_for(wl2)
    ws = torch.empty(max(sva.remainder_workspace(p1), sva.remainder_workspace(p2)), dtype=torch.uint8,
                     device="cuda")
    outs = []
    for wl, prob in ((wl1, p1), (wl2, p2)):
        bits = inputs.generate(wl)
        dev = device_inputs(bits)
        nb = sva.num_blocks(prob)
        kept = _oracle_lists(wl, bits)
        idx, cnt = _arrays(kept, nb)
        qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
        o, _ = sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt, workspace=ws)
        fresh, _ = sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt)
        torch.cuda.synchronize()
        assert torch.equal(o, fresh), wl.name
        outs.append(o)
    assert outs[1].shape[2] == wl2.seq_len


@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_smaller_workspace_runs_head_groups(out_dtype):
    """A workspace for fewer (batch, head) pairs than the problem has: the call
    does the pairs in groups of as many as fit (here 2, 2, 2; 4, 2; 1 x 6) and
    must give exactly the one-pass result, output and LSE, whichever output
    type; below one pair's size the binding refuses."""
    wl = SC("rem_groups", 2, 3, 128, (2, 6, 11), 64, "topk", keep_ratio=0.3, seed=311)
    prob = sva.problem_for(wl)
    if out_dtype == "f32":
        prob.out_dtype = 1
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    nb = sva.num_blocks(prob)
    kept = _oracle_lists(wl, bits)
    idx, cnt = _arrays(kept, nb)
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    full, full_lse = sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt,
                                                    want_lse=True)
    for heads in (2, 4, 1):
        ws = torch.empty(sva.remainder_workspace(prob, heads), dtype=torch.uint8, device="cuda")
        ws.fill_(0xFF)                                   # leftovers must not matter
        o, lse = sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt,
                                                want_lse=True, workspace=ws)
        torch.cuda.synchronize()
        say(f"[remainder groups] {out_dtype} {heads} pairs per pass")
        assert torch.equal(o, full) and torch.equal(lse, full_lse), heads
    small = torch.empty(sva.remainder_workspace(prob, 1) - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(ValueError):
        sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt, workspace=small)


def test_custom_softmax_scale():
    """A softmax scale other than 1/sqrt(D) reaches every place the remainder
    uses it: the first-order weights, the pooled-key logits and the c M q
    factor."""
    wl = SC("rem_scale", 1, 2, 64, (3, 10, 13), 64, "topk", keep_ratio=0.2, seed=310)
    c = 0.21
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl, out_dtype="f32", softmax_scale=c)
    nb = sva.num_blocks(prob)
    kept = _oracle_lists(wl, bits)
    idx, cnt = _arrays(kept, nb)
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    out, lse = sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt, want_lse=True)
    torch.cuda.synchronize()
    got, glse = out.cpu().numpy(), lse.cpu().numpy()
    for h in range(wl.heads):
        f = {n: oracle.bf16_bits_to_f64(bits[n][0, h])[None, None] for n in ("q", "k", "v")}
        ref, rlse = orem.remainder_attention(f["q"], f["k"], f["v"], [[kept[0][h]]], wl.block, c,
                                             weight=parity.KERNEL_REMAINDER_FORM)
        ref0, _ = orem.remainder_attention(f["q"], f["k"], f["v"], [[kept[0][h]]], wl.block, c, first_order=False,
                                           weight=parity.KERNEL_REMAINDER_FORM)
        excess, mean, mean_bound = parity.remainder_errors(got[0, h], ref[0, 0], ref[0, 0] - ref0[0, 0], False)
        assert excess <= 0.0 and mean <= mean_bound, (h, excess, mean, mean_bound)
        bound = parity.remainder_lse_bound(f["q"][0, 0], oracle.pool_blocks(f["k"][0, 0], wl.block), c)
        assert np.all(np.abs(glse[0, h] - rlse[0, 0]) <= bound), h
        # and the scale matters: the result at 1/sqrt(D) is far from this one
        other, _ = orem.remainder_attention(f["q"], f["k"], f["v"], [[kept[0][h]]], wl.block, scale_of(wl),
                                            weight=parity.KERNEL_REMAINDER_FORM)
        assert np.abs(other[0, 0] - ref[0, 0]).max() > 10 * parity.MAX_ABS
