"""Paged KV-cache write, written out from its definition.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``): only the tests, smoke() and
the bench's CPU-baseline leg may use it.

The serving engine the paper builds on (Sec. "Implementation": vLLM, whose KV
cache is paged -- PagedAttention) keeps each token's keys and values in fixed
16-token pages; a token is placed by its slot, slot = page * 16 + offset.
Writing a batch of new tokens (a prefill's prompt tokens, or one decode step's
token per sequence) copies token t's K and V, for every kv head, into
``cache[slot // 16, head, slot % 16, :]``.  Tokens whose slot is negative
(padding) are not written.  Nothing else in the cache changes.

Works on bf16 bit patterns (numpy uint16) or any dtype: it is a pure copy.
"""
from __future__ import annotations

import numpy as np


def write_kv_cache(k_cache, v_cache, k, v, slot_mapping, block_size: int = 16):
    """Return new (k_cache, v_cache) with the tokens of k, v ([T, Hkv, d])
    stored at their slots; the inputs are not modified.

    k_cache, v_cache: [num_blocks, Hkv, block_size, d]; slot_mapping: int [T].
    """
    kc = np.array(k_cache, copy=True)
    vc = np.array(v_cache, copy=True)
    k = np.asarray(k)
    v = np.asarray(v)
    slots = np.asarray(slot_mapping, dtype=np.int64)
    assert k.shape == v.shape and k.ndim == 3 and slots.shape == (k.shape[0],)
    for t in range(k.shape[0]):
        slot = int(slots[t])
        if slot < 0:
            continue
        page, offset = divmod(slot, block_size)
        kc[page, :, offset, :] = k[t]
        vc[page, :, offset, :] = v[t]
    return kc, vc


def slots_from_block_table(block_table_row, positions, block_size: int = 16):
    """Slots of the token positions of one sequence whose logical pages are
    block_table_row: position j lives in page block_table_row[j // 16] at
    offset j % 16."""
    pos = np.asarray(positions, dtype=np.int64)
    row = np.asarray(block_table_row, dtype=np.int64)
    return row[pos // block_size] * block_size + pos % block_size
