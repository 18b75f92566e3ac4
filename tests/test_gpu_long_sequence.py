"""One very long sequence, beyond the workloads' 35,904-token prompts: a
causal prefill of 131,109 tokens (GQA 8:1, d = 128; several thousand key
tiles per query tile, row offsets past 2^17) and one paged decode step over
131,110 keys (the 64-split maximum of the split-KV merge).  Sampled rows, all
heads, against the fp64 oracle."""
import numpy as np
import pytest
import torch

import gpu_support as G
from paper_2412_10543_amd import binding
from paper_2412_10543_amd.workloads import bf16_bits, normal_bf16

pytestmark = pytest.mark.gpu

L, HQ, HKV, D = 131072 + 37, 8, 1, 128


def test_prefill_very_long_sequence(orc):
    q = normal_bf16((L, HQ, D), 501, "cuda")
    k = normal_bf16((L, HKV, D), 502, "cuda")
    v = normal_bf16((L, HKV, D), 503, "cuda")
    o = torch.empty_like(q)
    cu = G.to_dev_i32([0, L])
    binding.rag_attn_prefill_varlen(q, k, v, o, None, cu, cu, L, L, G.scale_for(D), True)
    torch.cuda.synchronize()
    rng = np.random.Generator(np.random.PCG64(5))
    rows = sorted({0, 1, 63, 64, 65535, 65536, 131071, L - 2, L - 1} |
                  {int(x) for x in rng.integers(0, L, size=7)})
    rr = [r for r in rows for _ in range(HQ)]
    hh = [h for _ in rows for h in range(HQ)]
    want, _ = G.oracle_seq_rows(orc, q, bf16_bits(k), bf16_bits(v), L, rr, hh, G.scale_for(D))
    got = o[torch.as_tensor(rr).long().cuda(), torch.as_tensor(hh).long().cuda()]
    G.assert_parity(got.float().cpu().numpy(), want, "131k-token prefill")


def test_decode_very_long_sequence(orc):
    q, pool = G.decode_case([L + 1], HQ, HKV, D, seed=504)
    assert binding.rag_attn_decode_num_splits(1, HKV, pool.block_tables.shape[1]) == 64
    o = G.gpu_paged(q, pool, HQ, HKV, D, G.scale_for(D))
    G.assert_parity(o, G.oracle_paged(orc, q, pool, G.scale_for(D)), "131k-key decode")
