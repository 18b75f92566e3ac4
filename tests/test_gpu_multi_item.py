"""Prefill workgroups that run several query tiles ("items") one after another,
forced on small shapes with RAG_ATTN_PF_ITEMS, against the fp64 oracle (full
output, all heads, LSE) and bit for bit against one item per workgroup.

With items > 1 the kernel overlaps each item's start with the end of the one
before (next Q and first K/V tile copied into retired stages, early Q copies
for items of one or two key tiles, stage rotation, output staged through a
retired stage); the load-balancing choice only picks items > 1 for batches
with more than 8192 (stream, query tile) pairs, so these small cases are the
element-wise check of that path.  In the snake order a workgroup's first item
is its smallest tile (one or two key tiles for workgroups 0 and 1), followed
by longer ones, and ragged batches leave later items without rows."""
import os

import numpy as np
import pytest
import torch

import gpu_support as G

pytestmark = pytest.mark.gpu


def _with_items(n, fn):
    old = os.environ.get("RAG_ATTN_PF_ITEMS")
    os.environ["RAG_ATTN_PF_ITEMS"] = str(n)
    try:
        return fn()
    finally:
        if old is None:
            del os.environ["RAG_ATTN_PF_ITEMS"]
        else:
            os.environ["RAG_ATTN_PF_ITEMS"] = old


CASES = [
    # (q lengths, k lengths, hq, hkv, d)
    ([576] * 6, [576] * 6, 32, 8, 128),                      # map_reduce mappers
    ([640, 1, 65, 300, 0, 129, 511], None, 8, 2, 128),       # ragged, empty, 1-row
    ([1000, 64, 200], None, 4, 2, 64),
    ([450, 128], None, 8, 8, 128),                           # MHA (G = 1)
    ([700], None, 16, 2, 128),                               # G = 8: two head groups
    ([40, 300, 90], [300, 900, 90], 8, 2, 128),               # suffix rows (bottom-right)
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_multi_item_prefill(orc, case):
    lq, lk, hq, hkv, d = CASES[case]
    lk = lq if lk is None else lk
    q, k, v = G.prefill_inputs(lq, lk, hq, hkv, d, seed=900 + case)
    sc = G.scale_for(d)
    o1, l1 = _with_items(1, lambda: G.gpu_prefill(q, k, v, lq, lk, sc))
    ro, rl = G.oracle_prefill(orc, q, k, v, lq, lk, sc)
    fin = np.isfinite(rl)
    for items in (2, 3, 5, 32):
        print(f"multi-item case {case} items {items}: lq={lq} lk={lk} hq={hq} hkv={hkv} d={d}",
              flush=True)
        on, ln = _with_items(items, lambda: G.gpu_prefill(q, k, v, lq, lk, sc))
        assert torch.equal(on.view(torch.int16), o1.view(torch.int16)), \
            f"items={items}: output differs from items=1"
        assert torch.equal(ln, l1), f"items={items}: lse differs from items=1"
        G.assert_parity(on, ro, f"items={items}")
        got = ln.cpu().numpy()
        assert np.array_equal(np.isfinite(got), fin)
        assert np.max(np.abs(got[fin] - rl[fin]), initial=0.0) < 1e-3, "lse"


def test_multi_item_noncausal_and_peaky(orc):
    lq = [300, 200, 64]
    q, k, v = G.prefill_inputs(lq, lq, 8, 2, 128, seed=990, q_scale=6.0)
    sc = G.scale_for(128)
    for causal in (True, False):
        o, _ = _with_items(4, lambda: G.gpu_prefill(q, k, v, lq, lq, sc, causal=causal))
        ro, _ = G.oracle_prefill(orc, q, k, v, lq, lq, sc, causal=causal)
        G.assert_parity(o, ro, f"causal={causal}")
