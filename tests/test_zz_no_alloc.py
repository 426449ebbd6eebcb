"""The allocation-free token selection (sva_token_select_noalloc) against
sva_token_select with a caller workspace: bit-equal scores, kept indices and
positions on two calls in a row, the second on a smaller input (fewer batch
entries and tokens, so it runs over the first call's leftovers in the static
workspace), and a third at the largest batch the static workspace holds.
Outputs are allocated before the calls, so nothing is allocated around them.
"""
import ctypes

import pytest

import paper_2606_23743_amd as sva
from paper_2606_23743_amd import _lib, inputs

from .gpu_cases import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _outputs(B, N, k):
    return (torch.empty((B, N), dtype=torch.float64, device="cuda"),
            torch.empty((B, k), dtype=torch.int32, device="cuda"),
            torch.empty((B, N), dtype=torch.int32, device="cuda"))


@pytest.mark.parametrize("first,second", [((3, 20000, 512, 0.5), (1, 1500, 64, 0.3))])
def test_noalloc_matches_workspace_form(first, second):
    lib = _lib.load()
    stream = torch.cuda.current_stream().cuda_stream
    for B, N, C, r in (first, second, (16, 700, 128, 0.5)):
        x = inputs.to_device(inputs.hidden_states(B, N, C, seed=500 + B), "cuda")
        t = sva.tokens(B, N, C)
        k = sva.token_keep_count(t, r)
        want = _outputs(B, N, k)
        got = _outputs(B, N, k)
        ws = torch.empty(sva.token_select_workspace(t), dtype=torch.uint8, device="cuda")
        for o in got:
            o.fill_(-7)                                   # stale values must all be overwritten
        torch.cuda.synchronize()
        say(f"[no-alloc] B={B} N={N} C={C} k={k}")
        st = lib.sva_token_select(ctypes.byref(t), float(r), x.data_ptr(), want[0].data_ptr(), want[1].data_ptr(),
                                  want[2].data_ptr(), ws.data_ptr(), ws.numel(), stream)
        assert st == _lib.SVA_OK, st
        st = lib.sva_token_select_noalloc(ctypes.byref(t), float(r), x.data_ptr(), got[0].data_ptr(),
                                          got[1].data_ptr(), got[2].data_ptr(), stream)
        assert st == _lib.SVA_OK, st
        torch.cuda.synchronize()
        for a, b in zip(want, got):
            assert torch.equal(a, b), (B, N, C)
    # more batch entries than the static workspace holds: refused, nothing launched
    x = torch.zeros((17, 64, 8), dtype=torch.bfloat16, device="cuda")
    o = _outputs(17, 64, 32)
    t = sva.tokens(17, 64, 8)
    assert lib.sva_token_select_noalloc(ctypes.byref(t), 0.5, x.data_ptr(), o[0].data_ptr(), o[1].data_ptr(),
                                        o[2].data_ptr(), stream) == _lib.SVA_ERR_SHAPE
