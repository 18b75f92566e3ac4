"""Pins of the oracle's paged KV-cache write (oracle/kvcache.py), on the CPU.

The write is a pure copy, so every check is bit-exact: a brute-force
element-by-element copy, a round trip through block tables, the page layout of
the independent pool generator, untouched slots, skipped padding tokens, and
planted mistakes that the pins must catch.
"""
import numpy as np
import pytest

from oracle import slots_from_block_table, write_kv_cache
from paper_2412_10543_amd.workloads import bf16_bits, paged_pool


def _rand_bits(rng, shape):
    return rng.integers(0, 1 << 16, size=shape, dtype=np.uint16)


def _brute(k_cache, v_cache, k, v, slots):
    kc = k_cache.copy()
    vc = v_cache.copy()
    T, H, D = k.shape
    for t in range(T):
        if slots[t] < 0:
            continue
        for h in range(H):
            for d in range(D):
                kc[slots[t] // 16, h, slots[t] % 16, d] = k[t, h, d]
                vc[slots[t] // 16, h, slots[t] % 16, d] = v[t, h, d]
    return kc, vc


@pytest.mark.parametrize("T,H,D,nb", [(1, 1, 8, 1), (5, 2, 8, 3), (33, 3, 16, 5), (0, 2, 8, 2)])
def test_brute_force(T, H, D, nb):
    rng = np.random.Generator(np.random.PCG64(T * 31 + H))
    kc = _rand_bits(rng, (nb, H, 16, D))
    vc = _rand_bits(rng, (nb, H, 16, D))
    k = _rand_bits(rng, (T, H, D))
    v = _rand_bits(rng, (T, H, D))
    slots = rng.permutation(nb * 16)[:T].astype(np.int32)
    if T > 2:
        slots[1] = -1
    got = write_kv_cache(kc, vc, k, v, slots)
    want = _brute(kc, vc, k, v, slots)
    assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])


def test_round_trip_and_untouched_slots():
    """Writing each sequence's tokens at the slots its block table gives, then
    reading them back through the table, returns them exactly; every other
    slot keeps its previous bits."""
    rng = np.random.Generator(np.random.PCG64(5))
    H, D = 2, 8
    lens = [1, 16, 17, 40]
    nblk = [(n + 15) // 16 for n in lens]
    num_blocks = sum(nblk) + 3
    perm = rng.permutation(num_blocks)
    tables, pos = [], 0
    for nb in nblk:
        tables.append(perm[pos:pos + nb])
        pos += nb
    kc = np.full((num_blocks, H, 16, D), 0x7FC1, dtype=np.uint16)   # NaN bits
    vc = np.full((num_blocks, H, 16, D), 0x7FC2, dtype=np.uint16)
    toks_k = [_rand_bits(rng, (n, H, D)) for n in lens]
    toks_v = [_rand_bits(rng, (n, H, D)) for n in lens]
    slots = np.concatenate([slots_from_block_table(tb, np.arange(n)) for tb, n in zip(tables, lens)])
    k2, v2 = write_kv_cache(kc, vc, np.concatenate(toks_k), np.concatenate(toks_v), slots)
    written = np.zeros((num_blocks, 16), dtype=bool)
    for tb, n, tk, tv in zip(tables, lens, toks_k, toks_v):
        j = np.arange(n)
        assert np.array_equal(k2[tb[j // 16], :, j % 16, :], tk)
        assert np.array_equal(v2[tb[j // 16], :, j % 16, :], tv)
        written[tb[j // 16], j % 16] = True
    untouched = ~written[:, None, :].repeat(H, axis=1)       # [block, head, slot]
    assert np.all(k2[untouched] == 0x7FC1) and np.all(v2[untouched] == 0x7FC2)


def test_agrees_with_pool_generator_layout():
    """The pool generator places token j of sequence s at block_tables[s][j//16],
    slot j%16, by its own code; writing the same tokens with the oracle into an
    empty cache reproduces the pool on every used slot."""
    lens = [3, 16, 29]
    pool = paged_pool(lens, 2, 64, seed=9, poison=True)
    kc, vc = bf16_bits(pool.k_cache), bf16_bits(pool.v_cache)
    table = pool.block_tables.numpy()
    ks, vs, slots = [], [], []
    for s, n in enumerate(lens):
        j = np.arange(n)
        ks.append(kc[table[s, j // 16], :, j % 16, :])
        vs.append(vc[table[s, j // 16], :, j % 16, :])
        slots.append(slots_from_block_table(table[s], j))
    empty_k = np.zeros_like(kc)
    empty_v = np.zeros_like(vc)
    k2, v2 = write_kv_cache(empty_k, empty_v, np.concatenate(ks), np.concatenate(vs),
                            np.concatenate(slots))
    for s, n in enumerate(lens):
        for j in range(n):
            b, o = table[s, j // 16], j % 16
            assert np.array_equal(k2[b, :, o], kc[b, :, o]) and np.array_equal(v2[b, :, o], vc[b, :, o])


def test_padding_tokens_skipped():
    rng = np.random.Generator(np.random.PCG64(11))
    kc = _rand_bits(rng, (2, 1, 16, 8))
    vc = _rand_bits(rng, (2, 1, 16, 8))
    k = _rand_bits(rng, (3, 1, 8))
    v = _rand_bits(rng, (3, 1, 8))
    k2, v2 = write_kv_cache(kc, vc, k, v, [-1, -5, -1])
    assert np.array_equal(k2, kc) and np.array_equal(v2, vc)


def _mutant_head_offset_swapped(k_cache, v_cache, k, v, slots):
    kc = k_cache.copy(); vc = v_cache.copy()
    for t, s in enumerate(slots):
        if s >= 0:   # [page, offset, head] instead of [page, head, offset]
            kc[s // 16].reshape(-1, kc.shape[-1])[(s % 16) * kc.shape[1]:(s % 16 + 1) * kc.shape[1]] = k[t]
            vc[s // 16].reshape(-1, vc.shape[-1])[(s % 16) * vc.shape[1]:(s % 16 + 1) * vc.shape[1]] = v[t]
    return kc, vc


def _mutant_offset_off_by_one(k_cache, v_cache, k, v, slots):
    kc = k_cache.copy(); vc = v_cache.copy()
    for t, s in enumerate(slots):
        if s >= 0:   # right page, offset one too far (wrapping inside the page)
            kc[s // 16, :, (s + 1) % 16] = k[t]
            vc[s // 16, :, (s + 1) % 16] = v[t]
    return kc, vc


@pytest.mark.parametrize("mutant", [_mutant_head_offset_swapped, _mutant_offset_off_by_one])
def test_planted_mistakes_are_caught(mutant):
    """The brute-force pin distinguishes plausible layout mistakes."""
    rng = np.random.Generator(np.random.PCG64(21))
    H, D, nb, T = 3, 8, 4, 40
    kc = _rand_bits(rng, (nb, H, 16, D)); vc = _rand_bits(rng, (nb, H, 16, D))
    k = _rand_bits(rng, (T, H, D)); v = _rand_bits(rng, (T, H, D))
    slots = rng.permutation(nb * 16)[:T]
    want = _brute(kc, vc, k, v, slots)
    got = mutant(kc, vc, k, v, slots)
    assert not (np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1]))
