"""taps_select_noalloc (the selection with the library's static scratch, for callers that
cannot allocate) against taps_select with a caller workspace, through the C ABI: bit-equal
trees, top-K lists and q_reach on two calls in a row, the second with a smaller input,
so that the second runs over what the first left in the shared array."""
import sys

import numpy as np
import pytest
import torch

from tests import _util as U
from workloads import BF16, gen_round

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def taps():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_00487_amd as taps
    taps.load()
    return taps


def _same(a, b):
    for name in ("parent", "token", "depth", "rank", "n_nodes", "topk_idx"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name
    assert torch.equal(a.q_reach.view(torch.int64), b.q_reach.view(torch.int64)), "q_reach"
    assert torch.equal(a.topk_val.view(torch.int32), b.topk_val.view(torch.int32)), "topk_val"


def test_noalloc_select_equals_workspace_select_twice(taps):
    for name in ("serve16", "qwen3_4b"):          # the second call is smaller
        print(f"[noalloc] {name}", flush=True)
        sys.stdout.flush()
        inp = gen_round(name, with_attention=False)
        c = inp.cfg
        sel = taps.Selector(c.batch, c.block, c.vocab, c.K, c.budget, dtype=c.dtype,
                            kind=c.kind, lambda1=c.lambda1, lambda2=c.lambda2, tau=c.tau,
                            beta=c.beta)
        assert sel.ws_bytes <= taps._lib.SELECT_SCRATCH_BYTES
        m = U.to_dev(inp.marginals, c.dtype == BF16)
        ref = sel(m)
        torch.cuda.synchronize()
        ref = taps.TreeBuffers(*[t.clone() for t in (ref.parent, ref.token, ref.depth, ref.rank,
                                                       ref.q_reach, ref.n_nodes, ref.topk_idx,
                                                       ref.topk_val)])
        got = taps.TreeBuffers.empty(c.batch, c.block, c.K, c.budget)
        for t in (got.parent, got.token, got.depth, got.rank, got.n_nodes, got.topk_idx):
            t.fill_(-7)
        sel.noalloc(m, got)
        torch.cuda.synchronize()
        _same(ref, got)
        U.assert_tree_equal(got, U.oracle_trees(inp), c)


def test_noalloc_rejects_selections_beyond_its_scratch(taps):
    """A selection whose workspace exceeds the static scratch is refused before anything is
    enqueued."""
    import ctypes
    lib = taps.load()
    p = taps._lib.SelectParams(4096, 32, 151936, 16, 64, BF16, 0, 1.0, 0.125, 0.0, 1.0, 0, None)
    assert lib.taps_select_workspace_bytes(ctypes.byref(p)) > taps._lib.SELECT_SCRATCH_BYTES
    tree = taps.TreeBuffers.empty(1, 1, 1, 1)
    st = tree.struct()
    marg = torch.empty(16, dtype=torch.uint8, device="cuda")
    rc = lib.taps_select_noalloc(marg.data_ptr(), ctypes.byref(p), ctypes.byref(st),
                                 torch.cuda.current_stream().cuda_stream)
    assert rc == taps._lib.TAPS_ERR_WORKSPACE
