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
