"""rag_attn_decode_paged_noalloc (the library's static per-device scratch in
place of a workspace) against rag_attn_decode_paged with a workspace, through
the C ABI: bit-identical outputs on consecutive calls of different shapes --
each call after a larger one, so the scratch holds the earlier call's partials
-- and within the fp64 oracle's tolerance; sizes beyond the scratch are
rejected before anything is enqueued."""
import numpy as np
import pytest
import torch

from gpu_support import (assert_parity, decode_case, gpu_paged, oracle_paged, scale_for,
                         to_dev_i32)
from paper_2412_10543_amd import binding
from paper_2412_10543_amd.workloads import normal_bf16, paged_pool

pytestmark = pytest.mark.gpu


def _noalloc(q, pool, scale, cu_q=None, num_decode=None, max_seqlen_q=1, num_splits=0):
    o = torch.full_like(q, float("nan"))
    binding.rag_attn_decode_paged_noalloc(
        q, pool.k_cache, pool.v_cache, o, pool.block_tables, to_dev_i32(pool.kv_lens), scale,
        cu_seqlens_q=None if cu_q is None else to_dev_i32(cu_q), num_decode_seqs=num_decode,
        max_seqlen_q=max_seqlen_q, num_splits=num_splits)
    torch.cuda.synchronize()
    return o


# (kv lengths, hq, hkv, d, splits): the second and third are smaller than the
# one before them; splits > 1 so that the scratch is used
CASES = [
    ([9000, 300, 4500, 77, 2600, 16, 1, 7000], 32, 8, 128, 0),
    ([700, 1234, 65], 16, 2, 64, 6),
    ([40, 17], 8, 8, 128, 3),
]


def test_noalloc_matches_workspace_entry_on_consecutive_calls(orc):
    for rep in range(2):
        for i, (lens, hq, hkv, d, splits) in enumerate(CASES):
            print(f"noalloc case {i} rep {rep}: {len(lens)} seqs hq={hq} hkv={hkv} d={d} "
                  f"splits={splits}", flush=True)
            n = binding.rag_attn_decode_num_splits(len(lens), hkv, max((x + 15) // 16 for x in lens),
                                                   16, splits)
            assert n > 1
            q, pool = decode_case(lens, hq, hkv, d, 4100 + 10 * i)
            want = gpu_paged(q, pool, hq, hkv, d, scale_for(d), num_splits=splits)
            got = _noalloc(q, pool, scale_for(d), num_splits=splits)
            assert torch.equal(got.view(torch.int16), want.view(torch.int16)), f"case {i}"
            if rep == 0:
                assert_parity(got, oracle_paged(orc, q, pool, scale_for(d)), f"case {i}")


def test_noalloc_mixed_batch(orc):
    """Decode rows and chunked-prefill pieces in one launch."""
    hq, hkv, d = 32, 8, 128
    dec = [3000, 40, 1500, 800]
    pieces = [(200, 900), (64, 64)]              # (query rows, kv length)
    lens = dec + [kv for _, kv in pieces]
    pool = paged_pool(lens, hkv, d, 4200, device="cuda")
    nq = [1] * len(dec) + [p for p, _ in pieces]
    cu = [0] + list(np.cumsum(nq))
    q = normal_bf16((cu[-1], hq, d), 4201, "cuda")
    kw = dict(cu_q=cu, num_decode=len(dec), max_seqlen_q=max(nq), num_splits=4)
    want = gpu_paged(q, pool, hq, hkv, d, scale_for(d), **kw)
    got = _noalloc(q, pool, scale_for(d), **kw)
    assert torch.equal(got.view(torch.int16), want.view(torch.int16))
    assert_parity(got, oracle_paged(orc, q, pool, scale_for(d), cu_q=cu), "mixed")


@pytest.mark.parametrize("num_seqs,hq,hkv,d,blocks,splits,what", [
    (4096, 32, 8, 128, 64, 64, "partials"),     # 4096*32*64*(128+1)*4 B > 32 MiB
    (16384, 8, 8, 64, 4, 2, "counters"),        # 131072 (row, kv head) counters
])
def test_noalloc_rejects_sizes_beyond_scratch(num_seqs, hq, hkv, d, blocks, splits, what):
    q = torch.zeros((num_seqs, hq, d), dtype=torch.bfloat16, device="cuda")
    o = torch.full_like(q, 7.0)
    kc = torch.zeros((blocks, hkv, 16, d), dtype=torch.bfloat16, device="cuda")
    table = torch.zeros((num_seqs, blocks), dtype=torch.int32, device="cuda")
    kv = torch.full((num_seqs,), blocks * 16, dtype=torch.int32, device="cuda")
    with pytest.raises(binding.RagError) as e:
        binding.rag_attn_decode_paged_noalloc(q, kc, kc, o, table, kv, scale_for(d),
                                              num_splits=splits)
    assert e.value.status == binding.RAG_ERR_WORKSPACE and "no-alloc" in str(e.value)
    torch.cuda.synchronize()
    assert bool((o == 7.0).all()), "a rejected call wrote its output"
