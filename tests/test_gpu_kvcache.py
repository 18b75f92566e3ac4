"""GPU parity of the paged KV-cache write (rag_kv_cache_write) against the
oracle's write, bit for bit, and the prefill -> cache -> decode path: a
prefill's packed K/V written into shuffled pages by the kernel, then the next
decode step appended and attended over those pages, against the fp64 oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2412_10543_amd import binding
from paper_2412_10543_amd.workloads import bf16_bits, normal_bf16

import gpu_support as G

pytestmark = pytest.mark.gpu


def _caches(num_blocks, hkv, d, seed, nan_fill=True):
    shape = (num_blocks, hkv, 16, d)
    kc = normal_bf16(shape, seed, "cuda")
    vc = normal_bf16(shape, seed + 1, "cuda")
    if nan_fill:
        kc[::3] = float("nan")
        vc[1::3] = float("nan")
    return kc, vc


@pytest.mark.parametrize("T,hkv,d,num_blocks,pad", [
    (1, 1, 64, 1, False), (17, 2, 64, 5, True), (300, 8, 128, 40, True),
    (1000, 8, 128, 80, False), (63, 4, 128, 4, True), (5000, 1, 128, 400, True)])
def test_kv_write_bit_exact(T, hkv, d, num_blocks, pad):
    rng = np.random.Generator(np.random.PCG64(T + hkv + d))
    kc, vc = _caches(num_blocks, hkv, d, T)
    k = normal_bf16((T, hkv, d), T + 7, "cuda")
    v = normal_bf16((T, hkv, d), T + 8, "cuda")
    slots = rng.permutation(num_blocks * 16)[:T].astype(np.int32)
    if pad:
        slots[rng.random(T) < 0.2] = -1
    want_k, want_v = oracle.write_kv_cache(bf16_bits(kc), bf16_bits(vc), bf16_bits(k),
                                           bf16_bits(v), slots)
    binding.rag_kv_cache_write(k, v, kc, vc, G.to_dev_i32(slots))
    torch.cuda.synchronize()
    assert np.array_equal(bf16_bits(kc), want_k)
    assert np.array_equal(bf16_bits(vc), want_v)


def test_kv_write_empty_batch():
    kc, vc = _caches(2, 2, 64, 3)
    before = bf16_bits(kc).copy()
    empty = torch.empty((0, 2, 64), dtype=torch.bfloat16, device="cuda")
    binding.rag_kv_cache_write(empty, empty, kc, vc, torch.empty(0, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    assert np.array_equal(bf16_bits(kc), before)


@pytest.mark.parametrize("lens,hq,hkv,d", [([300, 17, 1040], 32, 8, 128), ([64, 5], 4, 2, 64)])
def test_prefill_to_pages_to_decode(orc, lens, hq, hkv, d):
    """Prompt K/V go into shuffled pages through the kernel; the next token's
    K/V is appended the same way; decode over the pages matches the oracle's
    attention of the new token over the whole sequence."""
    rng = np.random.Generator(np.random.PCG64(sum(lens)))
    S = len(lens)
    full = [n + 1 for n in lens]                       # prompt + one decode token
    nblk = [(n + 15) // 16 for n in full]
    num_blocks = int(sum(nblk) * 1.25) + 1
    perm = rng.permutation(num_blocks)
    mb = max(nblk)
    table = np.zeros((S, mb), dtype=np.int32)
    pos = 0
    for s, nb in enumerate(nblk):
        table[s, :nb] = perm[pos:pos + nb]
        pos += nb
    kc, vc = _caches(num_blocks, hkv, d, 5)
    # prefill tokens, packed [T, Hkv, d], written by the kernel
    T = sum(lens)
    k = normal_bf16((T, hkv, d), 11, "cuda")
    v = normal_bf16((T, hkv, d), 12, "cuda")
    slots = np.concatenate([oracle.slots_from_block_table(table[s], np.arange(n))
                            for s, n in enumerate(lens)]).astype(np.int32)
    binding.rag_kv_cache_write(k, v, kc, vc, G.to_dev_i32(slots))
    # one decode token per sequence
    kn = normal_bf16((S, hkv, d), 13, "cuda")
    vn = normal_bf16((S, hkv, d), 14, "cuda")
    nslots = np.array([oracle.slots_from_block_table(table[s], [n])[0] for s, n in enumerate(lens)],
                      dtype=np.int32)
    binding.rag_kv_cache_write(kn, vn, kc, vc, G.to_dev_i32(nslots))
    q = normal_bf16((S, hq, d), 15, "cuda")
    o = torch.empty_like(q)
    ws = G.workspace_for(S, hq, hkv, d, mb)
    binding.rag_attn_decode_paged(q, kc, vc, o, torch.from_numpy(table).cuda(),
                                  G.to_dev_i32(full), G.scale_for(d), workspace=ws)
    torch.cuda.synchronize()
    # oracle: dense attention of the new token over prompt + itself
    cu = G.cu_from_lens(lens)
    kb, vb, knb, vnb = bf16_bits(k), bf16_bits(v), bf16_bits(kn), bf16_bits(vn)
    kd = np.concatenate([np.concatenate([kb[cu[s]:cu[s + 1]], knb[s:s + 1]]) for s in range(S)])
    vd = np.concatenate([np.concatenate([vb[cu[s]:cu[s + 1]], vnb[s:s + 1]]) for s in range(S)])
    ro, _ = orc.varlen(bf16_bits(q), kd, vd, list(range(S + 1)), G.cu_from_lens(full),
                       G.scale_for(d), True, want_lse=False)
    G.assert_parity(o, ro, "prefill -> pages -> decode")


# ---------------------------------------------------------------------------
# fused paths: the prompt prefill that fills the cache, the decode step that
# appends its token
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("items", [None, "1", "3"])
@pytest.mark.parametrize("lens,hq,hkv,d", [
    ([300, 17, 1040, 1, 64, 65], 32, 8, 128), ([64, 5, 129], 4, 2, 64), ([700, 33], 16, 2, 128),
    ([576] * 5, 8, 8, 128)])
def test_fused_prefill_cache_write(orc, lens, hq, hkv, d, items, monkeypatch):
    """Cache contents bit-exact with the oracle's write of the same slot
    mapping (some tokens skipped, pages shuffled, the rest of the pool NaN);
    attention output bit-identical to rag_attn_prefill_varlen and within the
    oracle's tolerance."""
    if items is not None:
        monkeypatch.setenv("RAG_ATTN_PF_ITEMS", items)
    rng = np.random.Generator(np.random.PCG64(sum(lens) + hq))
    T = sum(lens)
    num_blocks = (T + 15) // 16 * 2 + 3
    kc, vc = _caches(num_blocks, hkv, d, 21)
    q, k, v = G.prefill_inputs(lens, lens, hq, hkv, d, seed=31 + d)
    slots = rng.permutation(num_blocks * 16)[:T].astype(np.int32)
    slots[rng.random(T) < 0.1] = -1
    want_k, want_v = oracle.write_kv_cache(bf16_bits(kc), bf16_bits(vc), bf16_bits(k),
                                           bf16_bits(v), slots)
    cu = G.to_dev_i32(G.cu_from_lens(lens))
    o = torch.empty_like(q)
    lse = torch.empty((hq, T), dtype=torch.float32, device="cuda")
    binding.rag_attn_prefill_varlen_kvcache(q, k, v, o, lse, cu, max(lens), G.scale_for(d), kc, vc,
                                            G.to_dev_i32(slots))
    torch.cuda.synchronize()
    assert np.array_equal(bf16_bits(kc), want_k), "k_cache"
    assert np.array_equal(bf16_bits(vc), want_v), "v_cache"
    o_ref, lse_ref = G.gpu_prefill(q, k, v, lens, lens, G.scale_for(d))
    assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
    assert torch.equal(lse, lse_ref)
    ro, _ = G.oracle_prefill(orc, q, k, v, lens, lens, G.scale_for(d))
    G.assert_parity(o, ro, "fused prefill")


@pytest.mark.parametrize("splits", [1, 0, 3])
@pytest.mark.parametrize("kv_lens,hq,hkv,d", [
    ([1, 17, 500, 2049, 64, 16, 33], 32, 8, 128), ([1000, 3], 4, 2, 64), ([5000, 257], 16, 1, 128)])
def test_fused_decode_append(orc, kv_lens, hq, hkv, d, splits):
    """Each row's last key is the new token: written into its slot bit-exactly
    (the slot held NaN before), attended in the same launch -- output
    bit-identical to rag_kv_cache_write followed by rag_attn_decode_paged, and
    within the oracle's tolerance."""
    S = len(kv_lens)
    q, pool = G.decode_case(kv_lens, hq, hkv, d, seed=S * 7 + d)
    table = pool.block_tables.cpu().numpy()
    slots = np.array([oracle.slots_from_block_table(table[s], [n - 1])[0]
                      for s, n in enumerate(kv_lens)], dtype=np.int32)
    for s in slots:                                    # the new tokens' slots start as NaN
        pool.k_cache[s // 16, :, s % 16] = float("nan")
        pool.v_cache[s // 16, :, s % 16] = float("nan")
    kn = normal_bf16((S, hkv, d), 41, "cuda")
    vn = normal_bf16((S, hkv, d), 42, "cuda")
    kc0, vc0 = pool.k_cache.clone(), pool.v_cache.clone()
    want_k, want_v = oracle.write_kv_cache(bf16_bits(kc0), bf16_bits(vc0), bf16_bits(kn),
                                           bf16_bits(vn), slots)
    ws = G.workspace_for(S, hq, hkv, d, table.shape[1], splits)
    o = torch.empty_like(q)
    binding.rag_attn_decode_paged_append(q, kn, vn, pool.k_cache, pool.v_cache, o,
                                         pool.block_tables, G.to_dev_i32(kv_lens), G.scale_for(d),
                                         num_splits=splits, workspace=ws)
    torch.cuda.synchronize()
    assert np.array_equal(bf16_bits(pool.k_cache), want_k), "k_cache"
    assert np.array_equal(bf16_bits(pool.v_cache), want_v), "v_cache"
    # the same step as two calls: write, then decode
    binding.rag_kv_cache_write(kn, vn, kc0, vc0, G.to_dev_i32(slots))
    o2 = torch.empty_like(q)
    binding.rag_attn_decode_paged(q, kc0, vc0, o2, pool.block_tables, G.to_dev_i32(kv_lens),
                                  G.scale_for(d), num_splits=splits, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int16), o2.view(torch.int16))
    G.assert_parity(o, G.oracle_paged(orc, q, pool, G.scale_for(d)), "decode append")
