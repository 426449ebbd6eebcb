"""GPU parity of fp8 (e4m3) quantisation and attention against the oracle.

Quantisation decides integers (codes, exponents) from exact comparisons and
one float32 product (Q times the softmax scale in base 2) or subtraction (K
minus its smoothing vector), the same on both sides: codes, exponents and the
bf16 smoothing vector must be bit-equal.  Q's codes carry the softmax scale,
so the oracle's logits are ln(2) times the dequantised products.

Attention: the oracle computes softmax attention of the dequantised Q, K, V
in float64.  The GPU also rounds each unnormalised probability p to e4m3
before the PV product (l sums the same rounded weights), so
    O_gpu - O = -sum_m (p^_m - p_m)(V_m - O_gpu) / sum_m p_m,
a weighted sum of independent rounding errors.  Rounding to nearest with 3
mantissa bits errs by at most e = 2^-4 p in the normal range (2^-16 of the
row maximum among the subnormals, given the GPU's 2^6 offset), uniformly, so each term has standard deviation at most
e_m/sqrt(3) * |V_m - O|; a bf16 output adds its own rounding (2^-8 |O| at most).  The test predicts the RMS error of every output
element from the oracle's p and V and requires the observed RMS to stay below
twice that; the worst case, all errors aligned (sum of e_m |V_m - O| / l), is
checked per element.  The fp8 matrix instructions add their own summation
error (measured below 2e-4 of the sum of magnitudes), budgeted as 4e-3 p.
"""
import numpy as np
import pytest

import oracle
import oracle.fp8_attention as of8
import paper_2606_23743_amd as sva
from paper_2606_23743_amd import inputs, workloads

from . import fp8_bounds as fb
from .gpu_cases import device_inputs, oracle_pool_all, oracle_select, say, scale_of

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

E4M3 = np.array([of8.e4m3_value(c) for c in range(256)])


def _np(t):
    return t.cpu().numpy()


def _bf16_bits(t):
    return _np(t.view(torch.int16)).view(np.uint16)


def _check_quant(wl, bits, quant, heads=None):
    """Codes, exponents and the smoothing vector against the oracle (all heads,
    or the listed (b, h))."""
    B, H, N, D, S = wl.batch, wl.heads, wl.seq_len, wl.head_dim, wl.block
    DP = (D + 63) // 64 * 64                                  # code channels; D..DP-1 are zero
    heads = heads or [(b, h) for b in range(B) for h in range(H)]
    q8, k8, v8 = _np(quant["q8"]), _np(quant["k8"]), _np(quant["v8"])
    qe, ke, ve = _np(quant["q_exp"]), _np(quant["k_exp"]), _np(quant["v_exp"])
    km = _bf16_bits(quant["k_mean"])
    for b, h in heads:
        sl = slice(b, b + 1), slice(h, h + 1)
        x = {n: oracle.bf16_bits_to_f64(bits[n][sl]) for n in ("q", "k", "v")}
        ref = of8.quantize_qkv(x["q"], x["k"], x["v"], S, lam=of8.softmax_scale_log2(D))
        assert np.array_equal(qe[b, h], ref["q_exp"][0, 0]), (b, h)
        assert np.array_equal(ke[b, h], ref["k_exp"][0, 0]), (b, h)
        assert np.array_equal(ve[b, h, :D], ref["v_exp"][0, 0]) and not ve[b, h, D:].any(), (b, h)
        want_mean = oracle.bf16_bits_to_f64(km[b, h])
        assert np.array_equal(want_mean, ref["k_mean"][0, 0]), (b, h)
        assert np.array_equal(E4M3[q8[b, h, :N, :D]], ref["q_code"][0, 0]), (b, h)
        assert np.array_equal(E4M3[k8[b, h, :N, :D]], ref["k_code"][0, 0]), (b, h)
        assert not q8[b, h, N:].any() and not k8[b, h, N:].any()
        assert not q8[b, h, :, D:].any() and not k8[b, h, :, D:].any()
        vt = E4M3[v8[b, h]]                                   # [Np/64, DP, 64] -> [Np, DP]
        vt = vt.transpose(0, 2, 1).reshape(-1, DP)
        assert np.array_equal(vt[:N, :D], ref["v_code"][0, 0]), (b, h)
        assert not vt[N:].any() and not vt[:, D:].any()


def _dequantised(bits, S, b, h):
    x = {n: oracle.bf16_bits_to_f64(bits[n][b:b + 1, h:h + 1]) for n in ("q", "k", "v")}
    return of8.quantize_qkv(x["q"], x["k"], x["v"], S, lam=of8.softmax_scale_log2(x["q"].shape[-1]))


def _check_attention(got, got_lse, quant_ref, kept_row_lists, S, scale, rows, out_bf16=True):
    """got: [N, D] float64 GPU output of one head; rows: query block ids to check;
    scale: the logit scale of the dequantised products (LN2: Q carries the
    softmax scale in base 2).
    Per weight p (oracle units, row maximum 1) the GPU's rounding errs by at
    most e = max(2^-4 p, min(p, 2^-16)): 3 mantissa bits, and e4m3 spacing
    2^-9 below 2^-6, where the GPU holds p times 2^(6 + k), 0 <= k <= 2.75
    (its probabilities are offset by 2^6 from a reference within 2.75 of the
    row maximum); plus 4e-3 p for the float32 summation inside the fp8
    instructions.  A bf16 output adds its own rounding, at most half an ulp
    (2^-8 |O|) and uniform: variance (2^-8 |O|)^2 / 3 per element.  Returns
    (observed rms, model rms)."""
    q, k, v = (quant_ref[n][0, 0] for n in ("q_hat", "k_hat", "v_hat"))
    N = q.shape[0]
    err2, pred2, cnt = 0.0, 0.0, 0
    for i in rows:
        qa, qb = i * S, min(N, (i + 1) * S)
        blocks = kept_row_lists[i]
        if not blocks:
            assert np.all(got[qa:qb] == 0)
            continue
        keys = np.concatenate([np.arange(j * S, min(N, (j + 1) * S)) for j in blocks])
        vk = v[keys]
        qstep = max(1, min(8, 20_000_000 // (len(keys) * vk.shape[1])))   # bounded host memory
        for q0 in range(qa, qb, qstep):
            q1 = min(qb, q0 + qstep)
            logits = scale * (q[q0:q1] @ k[keys].T)
            mx = logits.max(axis=1, keepdims=True)
            p = np.exp(logits - mx)
            l = p.sum(axis=1, keepdims=True)
            o = (p @ vk) / l
            lse = mx[:, 0] + np.log(l[:, 0])
            e = np.maximum(2.0 ** -4 * p, np.minimum(p, 2.0 ** -16)) + 4e-3 * p
            dev = np.abs(vk[None, :, :] - o[:, None, :])                # [q, m, D]
            bound = (e[:, :, None] * dev).sum(axis=1) / l + 2.0 ** -8 * np.abs(o) + 1e-6
            d = got[q0:q1] - o
            assert np.all(np.abs(d) <= bound), (i, float((np.abs(d) - bound).max()))
            var = ((e * e / 3.0)[:, :, None] * dev * dev).sum(axis=1) / (l * l)
            if out_bf16:
                var = var + (2.0 ** -8 * o) ** 2 / 3.0
            pred2 += float(var.sum())
            err2 += float((d * d).sum())
            cnt += d.size
            lbound = np.log1p(e.sum(axis=1) / l[:, 0]) + 1e-5
            assert np.all(np.abs(got_lse[q0:q1] - lse) <= lbound), i
    return np.sqrt(err2 / cnt), np.sqrt(pred2 / cnt)


def _check_against_unquantised(got, bits, b, h, quant_ref, kept_row_lists, S, rows, out_bf16=True, queries=None):
    """The GPU's 8-bit attention (got: [N, D] of head (b, h)) against softmax
    attention of the unquantised bf16 inputs in float64.  Per element the
    error may reach the P-rounding worst case of _check_attention (taken on
    the dequantised values) plus SIGMAS standard deviations of the storage
    error model (tests/fp8_bounds.py: Q, K, V stored as e4m3 at their group
    scales) plus the bf16 output's rounding; the RMS over all checked
    elements must stay under twice the combined model.  queries: offsets
    inside each block to check (all when None).  Returns (mean |err|, max
    |err|, rms, model rms)."""
    x = {n: oracle.bf16_bits_to_f64(bits[n][b, h]) for n in ("q", "k", "v")}
    N, D = x["q"].shape
    c = 1.0 / np.sqrt(D)
    lam = of8.softmax_scale_log2(D)
    qf = of8.fold_scale(x["q"], lam)
    ks = (x["k"].astype(np.float32) - quant_ref["k_mean"][0, 0].astype(np.float32)).astype(np.float64)
    qh, kh, vh = (quant_ref[n][0, 0] for n in ("q_hat", "k_hat", "v_hat"))
    q_exp, k_exp, v_exp = (quant_ref[n][0, 0] for n in ("q_exp", "k_exp", "v_exp"))
    tok_block = np.arange(N) // S
    abs_sum, n_el, err_max, err2, pred2 = 0.0, 0, 0.0, 0.0, 0.0
    for i in rows:
        qa, qb = i * S, min(N, (i + 1) * S)
        blocks = kept_row_lists[i]
        if not blocks:
            continue
        keys = np.concatenate([np.arange(j * S, min(N, (j + 1) * S)) for j in blocks])
        qs = np.arange(qa, qb) if queries is None else np.array([qa + o for o in queries if qa + o < qb])
        step = max(1, min(8, 12_000_000 // (len(keys) * D)))
        for s0 in range(0, len(qs), step):
            qi = qs[s0:s0 + step]
            p, o, _ = fb.exact_attention(x["q"][qi], x["k"][keys], x["v"][keys], c)
            eq, ek, ev = fb.storage_errors(qf[qi], q_exp[tok_block[qi]], ks[keys], k_exp[tok_block[keys]],
                                           x["v"][keys], v_exp[:D])
            _, var_q = fb.quantisation_effect(qf[qi], eq, ks[keys], ek, x["v"][keys], ev, p, o)
            # P rounding and the fp8 products' summation, on the dequantised values
            ph, oh, _ = fb.exact_attention(qh[qi], kh[keys], vh[keys], of8.LN2)
            e = np.maximum(2.0 ** -4 * ph, np.minimum(ph, 2.0 ** -16)) + 4e-3 * ph
            dev = np.abs(vh[keys][None, :, :] - oh[:, None, :])
            bound_p = (e[:, :, None] * dev).sum(axis=1)
            var_p = ((e * e / 3.0)[:, :, None] * dev * dev).sum(axis=1)
            var = var_q + var_p + ((2.0 ** -8 * oh) ** 2 / 3.0 if out_bf16 else 0.0)
            d = got[qi] - o
            bound = bound_p + fb.SIGMAS * np.sqrt(var_q) + 2.0 ** -8 * np.abs(oh) + 1e-6
            assert np.all(np.abs(d) <= bound), (i, float((np.abs(d) - bound).max()))
            abs_sum += float(np.abs(d).sum())
            n_el += d.size
            err_max = max(err_max, float(np.abs(d).max()))
            err2 += float((d * d).sum())
            pred2 += float(var.sum())
    return abs_sum / n_el, err_max, np.sqrt(err2 / n_el), np.sqrt(pred2 / n_el)


CASES = [
    # (name, B, H, D, grid, S, keep)
    ("d128_s128_ragged", 1, 2, 128, (3, 5, 16), 128, 0.5),
    ("d128_s64", 1, 2, 128, (2, 6, 20), 64, 0.3),
    ("d64_s64_ragged", 2, 1, 64, (2, 7, 9), 64, 0.4),
    ("d64_s128", 1, 2, 64, (4, 4, 24), 128, 0.5),
    ("d128_s128_short", 1, 1, 128, (1, 1, 40), 128, 1.0),
    ("d112_s64_ragged", 1, 2, 112, (2, 7, 9), 64, 0.4),       # 112 channels carried as 128
    ("d112_s128", 2, 1, 112, (3, 4, 20), 128, 0.5),
]


@pytest.mark.parametrize("name,B,H,D,grid,S,keep", CASES, ids=[c[0] for c in CASES])
def test_fp8_quantise_and_attend(name, B, H, D, grid, S, keep):
    wl = workloads.small_case(name, B, H, D, grid, S, "topk", keep_ratio=keep, seed=61,
                              sink_tokens=32, sink_scale=3.0)
    say(f"[fp8 {name}]")
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    quant = sva.quantize_fp8(prob, dev["q"], dev["k"], dev["v"])
    torch.cuda.synchronize()
    _check_quant(wl, bits, quant)
    # kept lists from the oracle's own selection
    qp, kp = oracle_pool_all(bits, S)
    scores = oracle.block_scores(qp, kp, scale_of(wl))
    kept, _ = oracle_select(wl, scores)
    nb = oracle.num_blocks(wl.seq_len, S)
    kmax = max(1, max(len(r) for b in kept for h in b for r in h))
    idx, cnt = oracle.kept_to_arrays(kept, nb, kmax)
    idx_d = torch.from_numpy(np.ascontiguousarray(idx, dtype=np.int32)).cuda()
    cnt_d = torch.from_numpy(np.ascontiguousarray(cnt, dtype=np.int32)).cuda()
    out, lse = sva.sparse_attention_fp8(prob, quant, idx_d, cnt_d, want_lse=True)
    dout, dlse = sva.dense_attention_fp8(prob, quant, want_lse=True)
    torch.cuda.synchronize()
    o = _np(out.float()).astype(np.float64)
    do = _np(dout.float()).astype(np.float64)
    for b in range(B):
        for h in range(H):
            ref = _dequantised(bits, S, b, h)
            rows = range(nb)
            rms, pred = _check_attention(o[b, h], _np(lse)[b, h], ref, kept[b][h], S, of8.LN2, rows)
            assert rms <= 2.0 * pred + 5e-4, (b, h, rms, pred)
            drms, dpred = _check_attention(do[b, h], _np(dlse)[b, h], ref, [list(range(nb))] * nb, S,
                                           of8.LN2, rows)
            assert drms <= 2.0 * dpred + 5e-4, (b, h, drms, dpred)
            say(f"[fp8 {name}] b{b} h{h}: sparse rms {rms:.2e} (model {pred:.2e}), dense rms {drms:.2e} "
                f"(model {dpred:.2e})")
            # against attention of the unquantised inputs
            mean_u, max_u, rms_u, pred_u = _check_against_unquantised(o[b, h], bits, b, h, ref, kept[b][h], S,
                                                                      rows)
            assert rms_u <= 2.0 * pred_u, (b, h, rms_u, pred_u)
            say(f"[fp8 {name}] b{b} h{h} vs unquantised: mean |err| {mean_u:.2e}, max {max_u:.2e}, "
                f"rms {rms_u:.2e} (model {pred_u:.2e})")


@pytest.mark.parametrize("S,D,step", [(128, 128, 3.0), (128, 128, 40.0), (64, 128, 3.0), (64, 112, 40.0),
                                      (128, 64, -3.0)])
def test_fp8_guard_rescales_with_rising_logits(S, D, step):
    """Logits move by `step` (log2 units) from one kept block to the next.  Rising,
    every block's maximum exceeds the reference by more than the kernel's
    guard, so O and l are rescaled before its probabilities are formed (which
    would otherwise pass e4m3's largest value); falling, the later blocks'
    weights sink toward e4m3's subnormals.  Both must match the oracle."""
    nblk = 5
    wl = workloads.small_case(f"growth_{S}_{D}", 1, 1, D, (1, nblk * S // 16, 16), S, "topk", topk=nblk,
                              seed=41)
    bits = inputs.generate(wl)
    f = {n: inputs.bf16_bits_to_f32(bits[n]).copy() for n in ("q", "k", "v")}
    c = scale_of(wl)
    f["q"][0, 0] = 1.0
    for b in range(nblk):
        val = step * (b - nblk // 2) / (np.log2(np.e) * c * D)
        f["k"][0, 0, b * S:(b + 1) * S] = val + 0.05 * f["k"][0, 0, b * S:(b + 1) * S]
    new_bits = {n: inputs._round_bf16(f[n]) for n in f}
    dev = device_inputs(new_bits)
    prob = sva.problem_for(wl)
    quant = sva.quantize_fp8(prob, dev["q"], dev["k"], dev["v"])
    rows = [list(range(nblk)) for _ in range(nblk)]
    idx = torch.from_numpy(np.array(rows, dtype=np.int32).reshape(1, 1, nblk, nblk)).cuda()
    cnt = torch.from_numpy(np.full((1, 1, nblk), nblk, dtype=np.int32)).cuda()
    out, lse = sva.sparse_attention_fp8(prob, quant, idx, cnt, want_lse=True)
    torch.cuda.synchronize()
    o = _np(out.float()).astype(np.float64)
    assert np.isfinite(o).all()
    ref = _dequantised(new_bits, S, 0, 0)
    span = np.abs(ref["q_hat"][0, 0] @ ref["k_hat"][0, 0].T).max()      # base-2 logits
    assert span >= 1.9 * abs(step), span                      # the regime this test is about
    rms, pred = _check_attention(o[0, 0], _np(lse)[0, 0], ref, rows, S, of8.LN2, range(nblk))
    assert rms <= 2.0 * pred + 5e-4, (rms, pred)


@pytest.mark.parametrize("S,D,sign", [(128, 128, 1.0), (128, 128, -1.0), (64, 64, 1.0), (64, 112, -1.0)])
def test_fp8_far_logits_take_the_explicit_path(S, D, sign):
    """Base-2 logits near +-160, where exp2(s) alone would leave float32's
    range: block 0 at sign*160, four blocks at -sign*40 (K's mean stays zero,
    so smoothing keeps them).  With sign +1 every row's reference is near 160
    and the wave subtracts it before exp2; with sign -1 it starts near -160
    (the same explicit form), then the next block moves it to about 40 (O and
    l scaled by about 2^-200) and the scaled conversion takes over."""
    nblk = 5
    wl = workloads.small_case(f"far_{S}_{D}", 1, 1, D, (1, nblk * S // 16, 16), S, "topk", topk=nblk, seed=43)
    bits = inputs.generate(wl)
    f = {n: inputs.bf16_bits_to_f32(bits[n]).copy() for n in ("q", "k", "v")}
    c = scale_of(wl)
    f["q"][0, 0] = 1.0
    for b in range(nblk):
        val = sign * (160.0 if b == 0 else -40.0) / (np.log2(np.e) * c * D)
        f["k"][0, 0, b * S:(b + 1) * S] = val + 0.05 * f["k"][0, 0, b * S:(b + 1) * S]
    new_bits = {n: inputs._round_bf16(f[n]) for n in f}
    dev = device_inputs(new_bits)
    prob = sva.problem_for(wl)
    quant = sva.quantize_fp8(prob, dev["q"], dev["k"], dev["v"])
    rows = [list(range(nblk)) for _ in range(nblk)]
    idx = torch.from_numpy(np.array(rows, dtype=np.int32).reshape(1, 1, nblk, nblk)).cuda()
    cnt = torch.from_numpy(np.full((1, 1, nblk), nblk, dtype=np.int32)).cuda()
    out, lse = sva.sparse_attention_fp8(prob, quant, idx, cnt, want_lse=True)
    torch.cuda.synchronize()
    o = _np(out.float()).astype(np.float64)
    assert np.isfinite(o).all() and np.isfinite(_np(lse)).all()
    ref = _dequantised(new_bits, S, 0, 0)
    logits = ref["q_hat"][0, 0] @ ref["k_hat"][0, 0].T                 # base-2 logits
    assert np.abs(logits[:, :S]).min() > 120.0, np.abs(logits[:, :S]).min()   # the regime
    rms, pred = _check_attention(o[0, 0], _np(lse)[0, 0], ref, rows, S, of8.LN2, range(nblk))
    assert rms <= 2.0 * pred + 5e-4, (rms, pred)


def test_fp8_f32_output_and_empty_rows():
    wl = workloads.small_case("f32_empty", 1, 2, 128, (2, 4, 32), 128, "topk", keep_ratio=0.5, seed=67)
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    prob32 = sva.problem_for(wl)
    prob32.out_dtype = 1
    quant = sva.quantize_fp8(prob, dev["q"], dev["k"], dev["v"])
    nb = oracle.num_blocks(wl.seq_len, 128)
    idx = np.full((1, 2, nb, 2), -1, dtype=np.int32)
    cnt = np.zeros((1, 2, nb), dtype=np.int32)
    idx[0, 0, :, 0], cnt[0, 0, :] = 0, 1                       # head 0: block 0 only
    idx[0, 1, 1, :] = [7, 99]                                   # head 1 row 1: out of range -> empty
    cnt[0, 1, 1] = 2
    idx_d, cnt_d = torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda()
    o16, _ = sva.sparse_attention_fp8(prob, quant, idx_d, cnt_d)
    o32, lse = sva.sparse_attention_fp8(prob32, quant, idx_d, cnt_d, want_lse=True)
    torch.cuda.synchronize()
    assert o32.dtype == torch.float32
    assert torch.equal(o32.to(torch.bfloat16), o16)
    assert not o32[0, 1].any() and torch.all(torch.isinf(lse[0, 1]))   # no usable block: zeros, -inf
    ref = _dequantised(bits, 128, 0, 0)
    rms, pred = _check_attention(_np(o32[0, 0]).astype(np.float64), _np(lse)[0, 0], ref, [[0]] * nb, 128,
                                 of8.LN2, range(nb), out_bf16=False)
    assert rms <= 2.0 * pred + 1e-4


@pytest.mark.slow
def test_fp8_full_size_sampled():
    """The 64B-class layer: every head's Q exponents, two heads' codes and
    smoothing vectors, and sampled query blocks of three heads' attention
    (kept lists from the oracle's own selection on those heads), against the
    oracle."""
    wl = workloads.LARGE_64B
    say(f"[fp8 {wl.name}] generating")
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    quant = sva.quantize_fp8(prob, dev["q"], dev["k"], dev["v"])
    S, H, N = wl.block, wl.heads, wl.seq_len
    nb = oracle.num_blocks(N, S)
    sel = sva.select_for(wl)
    kmax = sva.max_keep(prob, sel)
    heads = (0, H // 2, H - 1)
    idx = np.full((1, H, nb, kmax), -1, dtype=np.int32)
    cnt = np.zeros((1, H, nb), dtype=np.int32)
    kept_h = {}
    for h in heads:
        qp = oracle.pool_blocks(oracle.bf16_bits_to_f64(bits["q"][0, h]), S)
        kp = oracle.pool_blocks(oracle.bf16_bits_to_f64(bits["k"][0, h]), S)
        sc = oracle.block_scores(qp, kp, scale_of(wl))
        kept = oracle.select_topk(sc, oracle.topk_count(nb, wl.keep_ratio, wl.topk))
        kept_h[h] = [list(r) for r in kept]
        for i, r in enumerate(kept_h[h]):
            idx[0, h, i, :len(r)] = sorted(r)
            cnt[0, h, i] = len(r)
    out, lse = sva.sparse_attention_fp8(prob, quant, torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda(),
                                        want_lse=True)
    torch.cuda.synchronize()
    say(f"[fp8 {wl.name}] checking")
    for h in (0, H - 1):
        _check_quant(wl, bits, quant, heads=[(0, h)])
    lam = of8.softmax_scale_log2(wl.head_dim)
    for h in range(H):
        x = of8.fold_scale(oracle.bf16_bits_to_f64(bits["q"][0, h]), lam)
        amax = [np.abs(x[i * S:min(N, (i + 1) * S)]).max() for i in range(nb)]
        assert np.array_equal(_np(quant["q_exp"])[0, h], [of8.scale_exponent(a) for a in amax]), h
    rng = np.random.default_rng(7)
    o = _np(out.float()).astype(np.float64)
    for h in heads:
        ref = _dequantised(bits, S, 0, h)
        rows = sorted(rng.choice(nb, 5, replace=False).tolist()) + [nb - 1]
        rms, pred = _check_attention(o[0, h], _np(lse)[0, h], ref, kept_h[h], S, of8.LN2, rows)
        say(f"[fp8 {wl.name}] head {h}: rms {rms:.2e} (model {pred:.2e})")
        assert rms <= 2.0 * pred + 5e-4
    del dev, quant, out, lse
    torch.cuda.empty_cache()


def test_fp8_full_size_against_unquantised():
    """The 64B-class layer on the GPU's own kept lists: 8-bit attention
    against softmax attention of the unquantised inputs on sampled query
    blocks (the first two and the last of three heads, three random ones, and
    the block holding the largest difference between the 8-bit and the bf16
    kernel over the whole layer), 32 queries of each (the block's first and
    last 16, and the token of the largest difference).  Per element within
    the derived bounds; the mean error is reported beside the 2e-3 bar the
    bf16 path meets."""
    wl = workloads.LARGE_64B
    say(f"[fp8 vs unquantised {wl.name}] generating")
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    S, H, N = wl.block, wl.heads, wl.seq_len
    nb = oracle.num_blocks(N, S)
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    idx, cnt, _ = sva.select_blocks(prob, sva.select_for(wl), qp, kp)
    quant = sva.quantize_fp8(prob, dev["q"], dev["k"], dev["v"])
    o8, _ = sva.sparse_attention_fp8(prob, quant, idx, cnt)
    o16, _ = sva.sparse_attention(prob, dev["q"], dev["k"], dev["v"], idx, cnt)
    torch.cuda.synchronize()
    diff = (o8.float() - o16.float()).abs()
    flat = int(torch.argmax(diff).item())
    hw, nw = (flat // (N * wl.head_dim)) % H, (flat // wl.head_dim) % N
    say(f"[fp8 vs unquantised {wl.name}] largest |fp8 - bf16| {diff.max().item():.3f} at head {hw} token {nw}; "
        f"mean {diff.mean().item():.2e}")
    del diff, o16, quant, qp, kp
    idx_h, cnt_h = _np(idx), _np(cnt)
    rng = np.random.default_rng(11)
    picks = {0: [0, 1, nb - 1], H // 2: [0, 1, nb - 1], H - 1: [0, 1, nb - 1]}
    for h in (0, H // 2, H - 1):
        picks[h] += rng.choice(np.arange(2, nb - 1), 1).tolist()
    picks.setdefault(hw, [])
    picks[hw].append(nw // S)
    o = _np(o8.float()).astype(np.float64)
    total, n_rows, worst = 0.0, 0, 0.0
    for h, rows in sorted(picks.items()):
        ref = _dequantised(bits, S, 0, h)
        kept_rows = {i: idx_h[0, h, i, :cnt_h[0, h, i]].tolist() for i in rows}
        lists = [kept_rows.get(i, []) for i in range(nb)]
        offs = list(range(16)) + list(range(S - 16, S))
        if h == hw and nw % S not in offs:
            offs.append(nw % S)                      # the token of the largest difference
        mean_u, max_u, rms_u, pred_u = _check_against_unquantised(o[0, h], bits, 0, h, ref, lists, S,
                                                                  sorted(set(rows)), queries=offs)
        assert rms_u <= 2.0 * pred_u, (h, rms_u, pred_u)
        say(f"[fp8 vs unquantised {wl.name}] head {h} blocks {sorted(set(rows))}: mean |err| {mean_u:.2e}, "
            f"max {max_u:.2e}, rms {rms_u:.2e} (model {pred_u:.2e})")
        total += mean_u
        n_rows += 1
        worst = max(worst, max_u)
    say(f"[fp8 vs unquantised {wl.name}] mean |err| over the sampled heads {total / n_rows:.2e} "
        f"(the bf16 path's bar: 2e-3), max {worst:.2e}")
    del dev, o8
    torch.cuda.empty_cache()
