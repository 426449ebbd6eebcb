"""Calls on a stream other than the current one.

The binding allocates workspaces (the remainder's, the token selection's) and
outputs on the current stream and launches on the stream it is given; it must
mark them as in use on that stream, or the caching allocator can hand a
workspace freed at return to the next allocation on the current stream while
the kernels still read and write it.  Here the side stream is held back by a
spin kernel, the calls are enqueued behind it and return, and the current
stream at once allocates blocks of the same sizes and keeps writing garbage
into them while the side stream's kernels run; the results must equal the same
calls made on the current stream.
"""
import numpy as np
import pytest

import paper_2606_23743_amd as sva
from paper_2606_23743_amd import inputs, workloads

from .gpu_cases import device_inputs, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _scribble(nbytes_list, rounds=64):
    """Allocate a block of each size on the current stream and overwrite it
    many times (one small kernel each), so the writes span the side stream's
    work."""
    blocks = [torch.empty(n, dtype=torch.uint8, device="cuda") for n in nbytes_list]
    for r in range(rounds):
        for b in blocks:
            b.fill_(0xFF if r % 2 else 0x7F)
    return blocks


def test_side_stream_workspaces_stay_private():
    wl = workloads.small_case("side_stream", 1, 2, 128, (4, 10, 13), 128, "topk", keep_ratio=0.2, seed=401)
    bits = inputs.generate(wl)
    dev = device_inputs(bits)
    prob = sva.problem_for(wl)
    sel = sva.select_for(wl)
    hb = inputs.hidden_states(2, 3000, 256, seed=402)
    x = inputs.to_device(hb, "cuda")

    # on the current stream: the reference results
    qp, kp = sva.pool_blocks(prob, dev["q"], dev["k"])
    idx, cnt, _ = sva.select_blocks(prob, sel, qp, kp)
    ref_rem, ref_lse = sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt,
                                                      want_lse=True)
    ref_sc, ref_ki, ref_kp = sva.token_select(x, 0.5)
    torch.cuda.synchronize()

    side = torch.cuda.Stream()
    ws_rem = sva.remainder_workspace(prob)
    ws_tok = sva.token_select_workspace(sva.tokens(2, 3000, 256))
    for trial in range(3):
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            torch.cuda._sleep(20_000_000)            # holds the side stream back (bounded spin)
        # allocated by the binding on the current stream, launched on `side`
        rem, lse = sva.sparse_attention_remainder(prob, dev["q"], dev["k"], dev["v"], qp, kp, idx, cnt,
                                                  want_lse=True, stream=side)
        sc, ki, kpos = sva.token_select(x, 0.5, stream=side)
        junk = _scribble([ws_rem, ws_tok, rem.numel() * 2, lse.numel() * 4])
        torch.cuda.synchronize()
        del junk
        assert torch.equal(rem, ref_rem) and torch.equal(lse, ref_lse), trial
        assert torch.equal(sc, ref_sc) and torch.equal(ki, ref_ki) and torch.equal(kpos, ref_kp), trial
    say("[streams] remainder and token selection on a side stream match the current-stream results")
    assert np.isfinite(ref_rem.float().cpu().numpy()).all()
