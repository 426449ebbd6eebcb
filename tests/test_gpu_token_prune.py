"""GPU parity of feat_norm token pruning (sva_token_select / _gather / _scatter)
against the oracle.

Scores are float64 sums of exact bf16 squares; the GPU and the oracle add them
in different orders, so they may differ by rounding: at most (C - 1) * 2^-53
of the score (a sum of non-negative terms).  Kept indices are integers decided
by those float64 sums: they must equal the oracle's, except that a token whose
oracle score lies within that rounding bound of the oracle's k-th largest score
may trade places with another such token (a near-tie that summation order can
flip).  Exact ties (bit-identical rows, zero rows) must resolve by index
exactly.  Gather and scatter move bytes: bit-exact, fed the oracle's indices.
"""
import numpy as np
import pytest

import oracle
import oracle.token_prune as otp
import paper_2606_23743_amd as sva
from paper_2606_23743_amd import inputs, workloads

from .gpu_cases import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

U = 2.0 ** -53


def _dev(bits):
    return inputs.to_device(bits)


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _oracle_scores(bits, chunk=4096):
    B, N, _ = bits.shape
    out = np.empty((B, N))
    for s0 in range(0, N, chunk):
        out[:, s0:s0 + chunk] = otp.token_scores(oracle.bf16_bits_to_f64(bits[:, s0:s0 + chunk]))
    return out


def _check_select(x_bits, keep_ratio, scores, kept_idx, kept_pos):
    B, N, C = x_bits.shape
    k = otp.keep_count(N, keep_ratio)
    ref_s = _oracle_scores(x_bits)
    got_s = scores.cpu().numpy()
    bound = (C - 1) * U * ref_s
    assert np.all(np.abs(got_s - ref_s) <= bound), float(np.max(np.abs(got_s - ref_s) - bound))
    ref_kept = otp.select_tokens(ref_s, k)
    got_kept = kept_idx.cpu().numpy().astype(np.int64)
    pos = kept_pos.cpu().numpy()
    n_swapped = 0
    for b in range(B):
        g = got_kept[b]
        assert np.all(np.diff(g) > 0) and g[0] >= 0 and g[-1] < N, "kept indices ascending, in range"
        # kept_pos is the inverse map of kept_idx, -1 elsewhere
        want_pos = np.full(N, -1, dtype=np.int64)
        want_pos[g] = np.arange(k)
        assert np.array_equal(pos[b], want_pos)
        if np.array_equal(g, ref_kept[b]):
            continue
        thr = np.sort(ref_s[b])[::-1][k - 1]
        diff = np.setxor1d(g, ref_kept[b])
        tol = 2 * (C - 1) * U * thr
        assert np.all(np.abs(ref_s[b, diff] - thr) <= tol), "only near-ties may trade places"
        n_swapped += len(diff)
    return n_swapped


SMALL = [
    # (name, B, N, C, keep_ratio)
    ("b2_n1000_c64_half", 2, 1000, 64, 0.5),
    ("b1_n1025_c512_ragged", 1, 1025, 512, 0.3),      # one past the selection workgroup
    ("b3_n5000_c136_tenth", 3, 5000, 136, 0.1),
    ("b1_n4097_c6144_wide", 1, 4097, 6144, 0.5),
    ("b2_n777_c8_keepall", 2, 777, 8, 1.0),
    ("b1_n300_c64_keepone", 1, 300, 64, 1e-9),
    ("b1_n1_c64_single", 1, 1, 64, 0.5),
]


@pytest.mark.parametrize("name,B,N,C,r", SMALL, ids=[c[0] for c in SMALL])
def test_select_gather_scatter_match_oracle(name, B, N, C, r):
    say(f"[token_prune {name}]")
    bits = inputs.hidden_states(B, N, C, seed=71 + N)
    x = _dev(bits)
    scores, kept_idx, kept_pos = sva.token_select(x, r)
    torch.cuda.synchronize()
    swapped = _check_select(bits, r, scores, kept_idx, kept_pos)
    assert swapped == 0, swapped          # no near-ties at these sizes (fixed seeds)

    # gather and scatter on the oracle's own indices: bit-exact
    k = otp.keep_count(N, r)
    ref_kept = otp.select_tokens(_oracle_scores(bits), k)
    idx_dev = torch.from_numpy(ref_kept.astype(np.int32)).cuda()
    xk = sva.token_gather(x, idx_dev)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(xk), otp.gather_tokens(bits, ref_kept))
    y = inputs.hidden_states(B, k, C, seed=5, dup_frac=0.0, n_zero=0)
    pos = np.full((B, N), -1, dtype=np.int32)
    for b in range(B):
        pos[b, ref_kept[b]] = np.arange(k)
    out = sva.token_scatter(_dev(y), torch.from_numpy(pos).cuda(), x)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(out), otp.scatter_tokens(y, ref_kept, bits))


def test_exact_ties_resolve_to_lower_index():
    """Every row identical: the first k tokens are kept; rows at two score
    levels with the cut inside the lower level: the lowest-index ones of it."""
    B, N, C = 2, 3000, 64
    row = inputs.hidden_states(1, 1, C, seed=3, dup_frac=0.0, n_zero=0)[0, 0]
    bits = np.broadcast_to(row, (B, N, C)).copy()
    hi = np.random.default_rng(4).choice(N, 700, replace=False)
    bits[1, hi] = inputs.hidden_states(1, 1, C, seed=9, dup_frac=0.0, n_zero=0)[0, 0]   # another row
    x = _dev(bits)
    scores, kept_idx, kept_pos = sva.token_select(x, 0.5)
    torch.cuda.synchronize()
    assert _check_select(bits, 0.5, scores, kept_idx, kept_pos) == 0
    assert np.array_equal(kept_idx.cpu().numpy()[0], np.arange(1500))


def test_ties_across_segments():
    """30000 tokens drawn from six rows: every score level is a wide tie that
    spans many selection segments and tiles; the cut falls inside one level."""
    B, N, C = 2, 30000, 64
    protos = inputs.hidden_states(1, 6, C, seed=23, dup_frac=0.0, n_zero=0)[0]
    pick = np.random.default_rng(24).integers(0, 6, size=(B, N))
    bits = np.ascontiguousarray(protos[pick])
    for r in (0.37, 0.5, 0.9):
        x = _dev(bits)
        scores, kept_idx, kept_pos = sva.token_select(x, r)
        torch.cuda.synchronize()
        assert _check_select(bits, r, scores, kept_idx, kept_pos) == 0, r


def test_in_place_scatter_and_round_trip():
    """select -> gather -> scatter of the unchanged rows returns the input, in
    place over a copy of it as well."""
    B, N, C = 2, 2500, 256
    bits = inputs.hidden_states(B, N, C, seed=17)
    x = _dev(bits)
    _, kept_idx, kept_pos = sva.token_select(x, 0.4)
    xk = sva.token_gather(x, kept_idx)
    out = sva.token_scatter(xk, kept_pos, x)
    base = torch.zeros_like(x)
    zero_base = sva.token_scatter(xk, kept_pos, base, out=base)   # in place
    torch.cuda.synchronize()
    assert torch.equal(out, x)
    kp = kept_pos.cpu().numpy()
    zb = _bits(zero_base)
    assert np.array_equal(zb[kp >= 0], bits[kp >= 0]) and not zb[kp < 0].any()


@pytest.mark.slow
def test_full_size_hidden_states():
    """The 64B-class token count with a 6144-wide hidden state (the video
    stream's Q heads laid out token-major): every score and every kept index
    against the oracle, gather and scatter checked row by row on a sample."""
    wl = workloads.LARGE_64B
    N, C = wl.seq_len, wl.heads * wl.head_dim
    say(f"[token_prune full] N={N} C={C}: generating")
    q = inputs.generate(wl)["q"]                                  # [1, H, N, D]
    bits = np.ascontiguousarray(q.transpose(0, 2, 1, 3).reshape(1, N, C))
    del q
    x = _dev(bits)
    scores, kept_idx, kept_pos = sva.token_select(x, 0.5)
    torch.cuda.synchronize()
    say("[token_prune full] select done; oracle scores")
    swapped = _check_select(bits, 0.5, scores, kept_idx, kept_pos)
    say(f"[token_prune full] near-tie swaps: {swapped}")
    xk = sva.token_gather(x, kept_idx)
    out = sva.token_scatter(xk, kept_pos, x)
    torch.cuda.synchronize()
    assert torch.equal(out, x)
    idx = kept_idx.cpu().numpy()[0]
    rows = np.random.default_rng(1).choice(len(idx), 64, replace=False)
    xkb = _bits(xk[0, torch.from_numpy(rows).cuda()])
    assert np.array_equal(xkb, bits[0, idx[rows]])
    del x, xk, out
    torch.cuda.empty_cache()
