"""Pins for the oracle's block scores and both selection rules.

Expectations come from hand-worked fixtures (tests/golden), closed forms, a
pure-Python sort with an explicit tie-break key, an independent cumsum-based
search for the mass rule, and invariants that any correct rule satisfies.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.cpu


def _golden(golden_dir):
    return json.load(open(os.path.join(golden_dir, "select_handworked.json")))


def test_scores_bruteforce_and_orientation():
    rng = np.random.default_rng(11)
    qp = rng.standard_normal((2, 5, 3))
    kp = rng.standard_normal((2, 5, 3))
    c = 0.37
    s = oracle.block_scores(qp, kp, c)
    for h in range(2):
        for i in range(5):
            for j in range(5):
                want = c * math.fsum(qp[h, i, d] * kp[h, j, d] for d in range(3))
                assert abs(s[h, i, j] - want) < 1e-14
    # rows are query blocks: swapping the roles of q and k transposes the matrix
    assert not np.allclose(s, np.swapaxes(s, -1, -2))


def test_golden_pool_then_topk(golden_dir):
    g = _golden(golden_dir)["pool_topk"]
    q = np.array(g["q_tokens"], dtype=np.float64)[None, None]
    k = np.array(g["k_tokens"], dtype=np.float64)[None, None]
    c = 1.0 / math.sqrt(g["head_dim"])
    s = oracle.block_scores(oracle.pool_blocks(q, g["block"]), oracle.pool_blocks(k, g["block"]), c)
    assert np.allclose(s[0, 0], c * np.array(g["raw_dots"]), rtol=0, atol=1e-15)
    assert oracle.select_topk(s, 2) == [[g["top2"]]]
    assert oracle.select_topk(s, 3) == [[g["top3"]]]


def test_golden_mass(golden_dir):
    g = _golden(golden_dir)["mass"]
    s = np.array([[math.log(5.0), math.log(2.0), 0.0, 0.0, 0.0]])
    for case in g["cases"]:
        got = oracle.select_cummass(s, case["tau"], case["cap"], case["forced"])
        assert got == [case["kept"]], case


@pytest.mark.parametrize("nb,ratio,topk,want", [
    (16, 0.0, 4, 4),        # tiny plumbing: explicit top-4
    (512, 0.25, 0, 128),    # 2B-class layer
    (872, 0.15, 0, 131),    # 64B-class layer: 130.8 -> 131
    (1182, 1.0, 0, 1182),   # CFG sweep ratios
    (1182, 0.5, 0, 591),
    (1182, 0.25, 0, 296),   # 295.5 -> 296
    (1182, 0.1, 0, 119),    # 118.2 -> 119
    (1180, 0.1, 0, 118),    # 0.1*1180 is 118.00000000000001 in binary64; the epsilon keeps 118
    (10, 0.01, 0, 1),       # never below one block
    (10, 0.0, 50, 10),      # never above nB
])
def test_topk_count_closed_form(nb, ratio, topk, want):
    assert oracle.topk_count(nb, ratio, topk) == want


def test_first_frame_and_cap_mid_layer():
    # 31x34x60 grid, S=64: frame 0 is tokens 0..2039, blocks 0..31 (block 31 straddles frames 0/1)
    f = oracle.first_frame_blocks(34, 60, 64, 989)
    assert f == list(range(32))
    assert oracle.mass_cap(989, 0.30, len(f)) == 297      # ceil(296.7)
    assert oracle.mass_cap(989, 0.01, len(f)) == 32       # never below |F|
    assert oracle.first_frame_blocks(16, 16, 64, 16) == [0, 1, 2, 3]


def _brute_topk_row(row, k):
    order = sorted(range(len(row)), key=lambda j: (-float(row[j]), j))
    return sorted(order[:k])


def test_topk_bruteforce_random_and_ties():
    rng = np.random.default_rng(5)
    s = rng.standard_normal((3, 4, 23))
    s[0, 0, 5] = s[0, 0, 17] = s[0, 0].max() + 1.0           # exact tie at the top
    s[1] = np.round(s[1])                                     # many exact ties
    for k in (1, 3, 7, 23):
        got = oracle.select_topk(s, k)
        for a in range(3):
            for i in range(4):
                assert got[a][i] == _brute_topk_row(s[a, i], k)
                assert len(got[a][i]) == k
    assert 5 in oracle.select_topk(s, 1)[0][0] and 17 not in oracle.select_topk(s, 1)[0][0]


def _independent_mass_row(s, tau, cap, forced):
    """Same rule via a different route: sort once, prefix sums, first index."""
    p = np.exp(s - s.max())
    p = p / p.sum()
    forced = sorted(set(forced))
    others = [j for j in sorted(range(len(s)), key=lambda j: (-s[j], j)) if j not in forced]
    m0 = sum(p[j] for j in forced)
    budget = cap - len(forced)
    if m0 >= tau or budget <= 0:
        return sorted(forced)
    csum = m0 + np.cumsum([p[j] for j in others])
    hit = np.nonzero(csum >= tau)[0]
    n_add = (hit[0] + 1) if hit.size else len(others)
    n_add = min(n_add, budget)
    return sorted(forced + others[:n_add])


@pytest.mark.parametrize("tau,cap_ratio,force", [(0.9, 0.3, True), (0.5, 1.0, False),
                                                 (0.99, 0.2, False), (0.9, 0.05, True)])
def test_mass_matches_independent_search_and_invariants(tau, cap_ratio, force):
    rng = np.random.default_rng(7)
    nb = 40
    s = 3.0 * rng.standard_normal((5, nb))
    forced = list(range(4)) if force else []
    cap = oracle.mass_cap(nb, cap_ratio, len(forced))
    got = oracle.select_cummass(s, tau, cap, forced)
    for r in range(5):
        kept = got[r]
        assert kept == _independent_mass_row(s[r], tau, cap, forced)
        p = np.exp(s[r] - s[r].max()); p /= p.sum()
        m = p[kept].sum()
        assert set(forced) <= set(kept)
        assert len(forced) <= len(kept) <= cap
        assert kept == sorted(set(kept))
        assert m >= tau - 1e-12 or len(kept) == cap
        added = [j for j in kept if j not in forced]
        if added:
            # the last block added (lowest-ranked) was needed: without it mass < tau
            last = min(added, key=lambda j: (s[r, j], -j))
            assert p[kept].sum() - p[last] < tau
            # everything not kept ranks below everything added
            dropped = [j for j in range(nb) if j not in kept]
            for j in dropped:
                assert (s[r, j], -j) < (s[r, last], -last)


def test_mass_uniform_closed_form():
    # equal scores: p = 1/nB each; with no forced blocks the count is ceil(tau*nB), the
    # lowest indices win the ties
    nb = 20
    s = np.zeros((1, nb))
    got = oracle.select_cummass(s, 0.87, nb, [])
    assert got == [list(range(18))]                 # 17 blocks give 0.85, 18 give 0.90


def test_mass_scale_matters_topk_does_not():
    rng = np.random.default_rng(9)
    qp = rng.standard_normal((1, 30, 8))
    kp = rng.standard_normal((1, 30, 8))
    a = oracle.block_scores(qp, kp, 1.0)
    b = oracle.block_scores(qp, kp, 0.1)
    assert oracle.select_topk(a, 5) == oracle.select_topk(b, 5)
    ma = oracle.select_cummass(a, 0.8, 30, [])
    mb = oracle.select_cummass(b, 0.8, 30, [])
    assert sum(map(len, ma[0])) < sum(map(len, mb[0]))   # flatter softmax keeps more blocks


def test_kept_arrays_and_mask():
    kept = [[[0, 2], [1]], [[3], []]]
    idx, cnt = oracle.kept_to_arrays(kept, 4, 3)
    assert idx.shape == (2, 2, 3) and cnt.tolist() == [[2, 1], [1, 0]]
    assert idx[0, 0].tolist() == [0, 2, -1] and idx[1, 1].tolist() == [-1, -1, -1]
    m = oracle.kept_to_mask(kept, 4)
    assert m[0, 0].tolist() == [1, 0, 1, 0] and m[1, 1].sum() == 0
    with pytest.raises(ValueError):
        oracle.kept_to_arrays([[0, 1, 2, 3]], 4, 3)
