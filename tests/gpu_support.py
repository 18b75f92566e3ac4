"""Helpers for the GPU parity tests: run the HIP path through the C ABI and the
fp64 oracle on the same seeded inputs, and compare.

The tolerance is the one the hot path is specified to: bf16 inputs, fp32
accumulation, max-abs error <= 2e-2 and mean-abs error <= 2e-3 against the
fp64 oracle.
"""
import contextlib
import math
import os

import numpy as np
import torch

from paper_2412_10543_amd import binding
from paper_2412_10543_amd.workloads import bf16_bits, normal_bf16, paged_pool

MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def cu_from_lens(lens):
    return [0] + list(np.cumsum(lens).astype(int))


def to_dev_i32(x):
    return torch.tensor(np.asarray(x, dtype=np.int32), dtype=torch.int32, device="cuda")


def errors(got, want):
    """got: GPU bf16 tensor (or float array); want: fp64 numpy."""
    g = got.float().cpu().numpy().astype(np.float64) if isinstance(got, torch.Tensor) else got
    w = np.asarray(want, dtype=np.float64)
    assert g.shape == w.shape, (g.shape, w.shape)
    assert np.all(np.isfinite(g)), "non-finite output"
    e = np.abs(g - w)
    return float(e.max()) if e.size else 0.0, float(e.mean()) if e.size else 0.0


def assert_parity(got, want, what=""):
    mx, mean = errors(got, want)
    assert mx <= MAX_ABS and mean <= MEAN_ABS, f"{what}: max {mx:.3e} mean {mean:.3e}"
    return mx, mean


# ---------------------------------------------------------------------------
# prefill
# ---------------------------------------------------------------------------
def prefill_inputs(lens_q, lens_k, hq, hkv, d, seed, q_scale=1.0, device="cuda"):
    tq, tk = int(sum(lens_q)), int(sum(lens_k))
    q = normal_bf16((tq, hq, d), seed, device, q_scale)
    k = normal_bf16((tk, hkv, d), seed + 1, device)
    v = normal_bf16((tk, hkv, d), seed + 2, device)
    return q, k, v


def gpu_prefill(q, k, v, lens_q, lens_k, scale, causal=True, want_lse=True):
    cu_q, cu_k = cu_from_lens(lens_q), cu_from_lens(lens_k)
    o = torch.empty_like(q)
    lse = torch.empty((q.shape[1], q.shape[0]), dtype=torch.float32, device="cuda") \
        if want_lse else None
    binding.rag_attn_prefill_varlen(q, k, v, o, lse, to_dev_i32(cu_q), to_dev_i32(cu_k),
                                    max(lens_q) if lens_q else 0, max(lens_k) if lens_k else 0,
                                    scale, causal)
    torch.cuda.synchronize()
    return o, lse


@contextlib.contextmanager
def env(name, value):
    """Sets a library knob read at each call (RAG_ATTN_PF_ITEMS,
    RAG_AWQ_SM_NB, RAG_AWQ_SM_SPLITS, ...) for the calls inside the block;
    None leaves it unset."""
    old = os.environ.get(name)
    if value is None:
        os.environ.pop(name, None)
    else:
        os.environ[name] = str(value)
    try:
        yield
    finally:
        if old is None:
            os.environ.pop(name, None)
        else:
            os.environ[name] = old


def oracle_prefill(orc, q, k, v, lens_q, lens_k, scale, causal=True):
    return orc.varlen(bf16_bits(q), bf16_bits(k), bf16_bits(v), cu_from_lens(lens_q),
                      cu_from_lens(lens_k), scale, causal)


# ---------------------------------------------------------------------------
# paged decode / mixed
# ---------------------------------------------------------------------------
def workspace_for(num_decode, hq, hkv, d, max_blocks, num_splits=0):
    n = binding.rag_attn_decode_workspace_size(num_decode, hq, hkv, d, max_blocks, 16,
                                               num_splits)
    return torch.zeros(max(n, 1), dtype=torch.uint8, device="cuda") if n else None


def gpu_paged(q, pool, hq, hkv, d, scale, cu_q=None, num_decode=None, max_seqlen_q=1,
              num_splits=0, kv_lens=None, stream=None):
    kl = pool.kv_lens if kv_lens is None else kv_lens
    ns = pool.block_tables.shape[0]
    nd = ns if cu_q is None else num_decode
    ws = workspace_for(nd, hq, hkv, d, pool.block_tables.shape[1], num_splits)
    o = torch.empty_like(q)
    binding.rag_attn_decode_paged(q, pool.k_cache, pool.v_cache, o, pool.block_tables,
                                  to_dev_i32(kl), scale,
                                  cu_seqlens_q=None if cu_q is None else to_dev_i32(cu_q),
                                  num_decode_seqs=nd, max_seqlen_q=max_seqlen_q,
                                  num_splits=num_splits, workspace=ws, stream=stream)
    torch.cuda.synchronize()
    return o


def oracle_paged(orc, q, pool, scale, cu_q=None, kv_lens=None):
    kl = pool.kv_lens if kv_lens is None else kv_lens
    o, _ = orc.paged(bf16_bits(q), bf16_bits(pool.k_cache), bf16_bits(pool.v_cache),
                     pool.block_tables.cpu().numpy(), kl, scale, cu_q=cu_q, want_lse=False)
    return o


def decode_case(kv_lens, hq, hkv, d, seed, q_scale=1.0):
    pool = paged_pool(kv_lens, hkv, d, seed, device="cuda")
    q = normal_bf16((len(kv_lens), hq, d), seed + 11, "cuda", q_scale)
    return q, pool


def scale_for(d):
    return 1.0 / math.sqrt(d)


# ---------------------------------------------------------------------------
# full-size workloads: sampled rows
# ---------------------------------------------------------------------------
def sample_rows(L, chunk_len, rng, n_random=16):
    """Row 0, the last row, both sides of every chunk boundary and seeded
    random rows of a prompt of L tokens."""
    rows = {0, L - 1}
    for b in range(chunk_len, L, chunk_len):
        rows.update((b - 1, b))
    rows.update(int(x) for x in rng.integers(0, L, size=n_random))
    return sorted(r for r in rows if 0 <= r < L)


def heads_for_row(row, hq, hkv):
    """One q head per kv group, rotating inside the group with the row."""
    g = hq // hkv
    return [kv * g + (row + kv) % g for kv in range(hkv)]


def dense_kv_of_seq(pool, s, n):
    """Keys and values 0..n-1 of sequence s gathered from the paged pool
    (test-side gather through the block table), as bf16 bit arrays
    [n, hkv, d]."""
    nb = (n + 15) // 16
    blocks = pool.block_tables[s, :nb].long()
    hkv, d = pool.k_cache.shape[1], pool.k_cache.shape[3]
    k = pool.k_cache[blocks].permute(0, 2, 1, 3).reshape(nb * 16, hkv, d)[:n]
    v = pool.v_cache[blocks].permute(0, 2, 1, 3).reshape(nb * 16, hkv, d)[:n]
    return bf16_bits(k), bf16_bits(v)


def oracle_seq_rows(orc, q_seq, k_bits, v_bits, nq, rows, heads, scale):
    """Oracle rows of one sequence.  q_seq: GPU tensor [nq, hq, d] of that
    sequence; rows/heads: parallel lists."""
    idx_r = torch.as_tensor(rows, device=q_seq.device).long()
    idx_h = torch.as_tensor(heads, device=q_seq.device).long()
    qr = bf16_bits(q_seq[idx_r, idx_h])
    o, lse = orc.seq_rows(qr, k_bits, v_bits, nq, np.asarray(rows), np.asarray(heads),
                          q_seq.shape[1], scale)
    return o, lse
