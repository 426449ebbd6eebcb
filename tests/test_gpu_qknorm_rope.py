"""GPU parity of the fused QKNorm + RoPE + pool producer (sva_qknorm_rope_pool)
against the oracle.

Outputs are bf16 computed in float32.  Turning a pair of norm r in float32
(two products and a sum, with sin and cos of the float64-reduced angle good to
3e-7) leaves an absolute error of at most about 4.5e-7 * r, and the RMSNorm
scale a relative 2^-22; so a written element may differ from the exact value's
bf16 rounding by one bf16 ulp of the result plus 2^-20 * r (9.5e-7 * r, twice
that bound; it matters only where a coordinate nearly cancels).  Elements that differ at all are those whose exact
value lies within that error of a rounding midpoint: at most MISMATCH_FRAC
(expected ~2^-12).  The block summaries must be exactly the float32-rounded
means of the GPU's own written outputs (and equal sva_pool_blocks on them).
"""
import numpy as np
import pytest

import oracle
import paper_2606_23743_amd as sva
from paper_2606_23743_amd import inputs, workloads

from .gpu_cases import device_inputs, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

MISMATCH_FRAC = 2e-3
EPS, BASE = 1e-6, 10000.0


def _ulp(x: np.ndarray) -> np.ndarray:
    _, e = np.frexp(x)
    return np.ldexp(1.0, np.maximum(e - 8, -133))


def _check_against_oracle(gpu_bits, exact, name):
    """exact: the oracle's unrounded float64 output."""
    ref = oracle.round_bf16(exact)
    got = oracle.bf16_bits_to_f64(gpu_bits)
    d = np.abs(got - ref)
    r = np.sqrt(exact[..., 0::2] ** 2 + exact[..., 1::2] ** 2)
    r = np.repeat(r, 2, axis=-1)
    assert np.all(d <= _ulp(ref) + 2.0 ** -20 * r), (name, float((d - _ulp(ref) - 2.0 ** -20 * r).max()))
    frac = float(np.count_nonzero(d)) / d.size
    assert frac <= MISMATCH_FRAC, (name, frac)
    return frac


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


CASES = [
    # (name, B, H, D, grid, S)
    ("d128_s128_ragged", 1, 2, 128, (3, 5, 16), 128),
    ("d112_s64_ragged", 2, 3, 112, (2, 7, 9), 64),
    ("d64_s64_short", 1, 2, 64, (1, 1, 40), 64),
    ("d128_s64", 1, 3, 128, (4, 6, 10), 64),
    ("d64_s128", 2, 1, 64, (5, 3, 20), 128),
    ("d128_s64_h10", 2, 10, 128, (2, 5, 13), 64),     # a full and a partial group of 8 heads
]


@pytest.mark.parametrize("name,B,H,D,grid,S", CASES, ids=[c[0] for c in CASES])
def test_producer_matches_oracle(name, B, H, D, grid, S):
    wl = workloads.small_case(name, B, H, D, grid, S, "topk", topk=1, seed=53)
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    rng = np.random.default_rng(11)
    gq = rng.uniform(0.5, 1.5, D).astype(np.float32)
    gk = rng.uniform(0.5, 1.5, D).astype(np.float32)
    prob = sva.problem_for(wl)
    qo, ko, qp, kp = sva.qknorm_rope_pool(prob, dev["q"], dev["k"], torch.from_numpy(gq).cuda(),
                                          torch.from_numpy(gk).cuda(), EPS, BASE)
    torch.cuda.synchronize()
    q64, k64 = (oracle.bf16_bits_to_f64(bits[n]) for n in ("q", "k"))
    rq = oracle.norm_rope(q64, gq.astype(np.float64), grid, EPS, BASE)
    rk = oracle.norm_rope(k64, gk.astype(np.float64), grid, EPS, BASE)
    fq = _check_against_oracle(_bits(qo), rq, "q")
    fk = _check_against_oracle(_bits(ko), rk, "k")
    # block summaries: the means of what was written
    for out, pooled, n in ((qo, qp, "q"), (ko, kp, "k")):
        want = oracle.pool_blocks(oracle.bf16_bits_to_f64(_bits(out)), S).astype(np.float32)
        assert np.array_equal(pooled.cpu().numpy(), want), n
    pq, pk = sva.pool_blocks(prob, qo, ko)
    torch.cuda.synchronize()
    assert torch.equal(pq, qp) and torch.equal(pk, kp)
    say(f"[producer {name}] ulp-off fraction q={fq:.2e} k={fk:.2e}")


def test_producer_in_place_equals_out_of_place():
    wl = workloads.small_case("inplace", 1, 2, 128, (2, 4, 24), 64, "topk", topk=1, seed=59)
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    g = torch.linspace(0.5, 1.5, 128, dtype=torch.float32, device="cuda")
    prob = sva.problem_for(wl)
    qo, ko, qp, kp = sva.qknorm_rope_pool(prob, dev["q"], dev["k"], g, g)
    q2, k2 = dev["q"].clone(), dev["k"].clone()
    qo2, ko2, qp2, kp2 = sva.qknorm_rope_pool(prob, q2, k2, g, g, q_out=q2, k_out=k2)
    torch.cuda.synchronize()
    assert qo2.data_ptr() == q2.data_ptr()
    assert torch.equal(qo, q2) and torch.equal(ko, k2) and torch.equal(qp, qp2) and torch.equal(kp, kp2)


@pytest.mark.slow
def test_producer_full_size_sampled_heads():
    """The 64B-class shape: every head's summaries equal sva_pool_blocks of the
    written tensors; two heads are checked against the oracle element by element."""
    wl = workloads.LARGE_64B
    say(f"[producer {wl.name}] generating")
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    D = wl.head_dim
    rng = np.random.default_rng(13)
    gq = rng.uniform(0.5, 1.5, D).astype(np.float32)
    gk = rng.uniform(0.5, 1.5, D).astype(np.float32)
    prob = sva.problem_for(wl)
    qo, ko, qp, kp = sva.qknorm_rope_pool(prob, dev["q"], dev["k"], torch.from_numpy(gq).cuda(),
                                          torch.from_numpy(gk).cuda(), EPS, BASE)
    pq, pk = sva.pool_blocks(prob, qo, ko)
    torch.cuda.synchronize()
    assert torch.equal(pq, qp) and torch.equal(pk, kp)
    grid = (wl.grid_t, wl.grid_h, wl.grid_w)
    for h in (0, wl.heads - 1):
        q64 = oracle.bf16_bits_to_f64(bits["q"][0:1, h:h + 1])
        k64 = oracle.bf16_bits_to_f64(bits["k"][0:1, h:h + 1])
        rq = oracle.norm_rope(q64, gq.astype(np.float64), grid, EPS, BASE)
        rk = oracle.norm_rope(k64, gk.astype(np.float64), grid, EPS, BASE)
        fq = _check_against_oracle(_bits(qo[0:1, h:h + 1]), rq, f"q head {h}")
        fk = _check_against_oracle(_bits(ko[0:1, h:h + 1]), rk, f"k head {h}")
        say(f"[producer {wl.name}] head {h}: ulp-off fraction q={fq:.2e} k={fk:.2e}")
    del dev, qo, ko, qp, kp, pq, pk
    torch.cuda.empty_cache()
