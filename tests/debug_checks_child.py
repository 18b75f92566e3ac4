"""Child process of test_gpu_debug_checks.py: run with RAG_ATTN_CHECK=1 in the
environment (the library reads it once per process), call each entry point
with valid device arrays and with arrays that break one documented
precondition, and print {case: status} as one JSON line.

In this mode the library copies the device index arrays to the host and
checks them before anything is enqueued, so the invalid cases never reach a
kernel.
"""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import torch  # noqa: E402

from paper_2412_10543_amd import binding  # noqa: E402
from paper_2412_10543_amd.workloads import normal_bf16, paged_pool  # noqa: E402

assert os.environ.get("RAG_ATTN_CHECK") == "1"
dev = torch.device("cuda:0")
i32 = lambda x: torch.tensor(x, dtype=torch.int32, device=dev)  # noqa: E731
out = {}


def run(name, fn):
    try:
        fn()
        torch.cuda.synchronize()
        out[name] = binding.RAG_OK
    except binding.RagError as e:
        out[name] = e.status


# ---- prefill: cu_seqlens must be monotone, within max_seqlen, nq <= nk (causal)
hq, hkv, d = 8, 2, 64
q = normal_bf16((100, hq, d), 1, dev)
k = normal_bf16((100, hkv, d), 2, dev)
v = normal_bf16((100, hkv, d), 3, dev)
o = torch.empty_like(q)
sc = d ** -0.5


def prefill(cq, ck, mq, mk, causal=True):
    return lambda: binding.rag_attn_prefill_varlen(q, k, v, o, None, i32(cq), i32(ck), mq, mk,
                                                   sc, causal)


run("prefill_valid", prefill([0, 40, 100], [0, 40, 100], 60, 60))
run("prefill_not_monotone", prefill([0, 50, 40], [0, 50, 40], 60, 60))
run("prefill_over_max_seqlen", prefill([0, 40, 100], [0, 40, 100], 50, 60))
run("prefill_more_rows_than_keys", prefill([0, 50, 100], [0, 40, 100], 60, 60))
run("prefill_suffix_rows", prefill([0, 10, 30], [0, 40, 100], 60, 60))

# ---- decode: 1 <= kv_len <= max_blocks*16, block ids in [0, num_blocks)
lens = [40, 300, 17]
pool = paged_pool(lens, hkv, d, 5, device=dev)
mb = pool.block_tables.shape[1]
qd = normal_bf16((len(lens), hq, d), 6, dev)
od = torch.empty_like(qd)
n_ws = binding.rag_attn_decode_workspace_size(len(lens), hq, hkv, d, mb)
ws = torch.zeros(max(n_ws, 256), dtype=torch.uint8, device=dev)


def decode(kv, table=None, cu_q=None, nd=None, mq=1, qq=None, oo=None, pl=None):
    pl = pool if pl is None else pl
    t = pl.block_tables if table is None else table
    return lambda: binding.rag_attn_decode_paged(
        qd if qq is None else qq, pl.k_cache, pl.v_cache, od if oo is None else oo, t,
        i32(kv), sc, cu_seqlens_q=None if cu_q is None else i32(cu_q), num_decode_seqs=nd,
        max_seqlen_q=mq, workspace=ws)


run("decode_valid", decode(lens))
run("decode_kv_len_zero", decode([40, 0, 17]))
run("decode_kv_len_past_table", decode([40, mb * 16 + 1, 17]))
bad = pool.block_tables.clone()
bad[1, 3] = pool.num_blocks
run("decode_block_id_too_large", decode(lens, bad))
bad = pool.block_tables.clone()
bad[2, 0] = -1
run("decode_block_id_negative", decode(lens, bad))
bad = pool.block_tables.clone()
bad[0, mb - 1] = pool.num_blocks     # past ceil(40/16) blocks: never read, not checked
run("decode_unused_entry_ignored", decode(lens, bad))

# mixed batch: decode rows have one query row; a piece has nq <= kv_len
mlens = [40, 300, 64]
mpool = paged_pool(mlens, hkv, d, 10, device=dev)
qm = normal_bf16((2 + 30, hq, d), 7, dev)
om = torch.empty_like(qm)
mixed = dict(nd=2, mq=30, qq=qm, oo=om, pl=mpool)
run("mixed_valid", decode(mlens, cu_q=[0, 1, 2, 32], **mixed))
run("mixed_decode_row_with_two_rows", decode(mlens, cu_q=[0, 2, 3, 32], **mixed))
run("mixed_piece_longer_than_keys", decode([40, 300, 20], cu_q=[0, 1, 2, 32], **mixed))

# ---- KV-cache write: slots unique and inside the pool; negative = padding
kc = torch.zeros((8, hkv, 16, d), dtype=torch.bfloat16, device=dev)
vc = torch.zeros_like(kc)
kn = normal_bf16((5, hkv, d), 8, dev)
vn = normal_bf16((5, hkv, d), 9, dev)


def write(slots):
    return lambda: binding.rag_kv_cache_write(kn, vn, kc, vc, i32(slots))


run("kv_write_valid", write([0, 17, 127, -1, 64]))
run("kv_write_duplicate_slot", write([0, 17, 17, -1, 64]))
run("kv_write_slot_past_pool", write([0, 17, 128, -1, 64]))

print(json.dumps(out), flush=True)
