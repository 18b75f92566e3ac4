"""The five workloads at full size, run in the configuration bench.py times
(same inputs, pools, workspace and split policy), against the fp64 oracle:

  prefill  tiny and mapred7b in full (every row, every head, and the LSE);
           stuff7b, long70b and the mixed batch's chunked-prefill pieces on a
           deterministic row sample with every head -- row 0, the last row,
           both sides of every chunk boundary and seeded random rows (1024 per
           prompt; 256 for long70b, whose 35,904-token prompts cost the fp64
           oracle ~2.4 TFLOP at 1024 rows);
  decode   every step of tiny, stuff7b and mapred7b (every sequence, every
           head); long70b at steps 0, 1, 127, 255 and 8 seeded random steps;
           the mixed batch's 256 decode rows.

A decode step t of a prompt of L tokens is row t of a "query block" of as many
rows as steps against the L + steps keys of its pool: row t sees L + t + 1
keys, so the oracle evaluates all steps of a sequence in one call.
Tolerance: max-abs 2e-2, mean-abs 2e-3."""
import numpy as np
import pytest
import torch

import bench
import gpu_support as G
import oracle
from paper_2412_10543_amd import binding
from paper_2412_10543_amd.workloads import bf16_bits, long70b, mapred7b, stuff7b, tiny

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

WORKLOADS = {"tiny": tiny, "stuff7b": stuff7b, "mapred7b": mapred7b, "long70b": long70b}
PREFILL_FULL = {"tiny", "mapred7b"}
RANDOM_ROWS = {"stuff7b": 1024, "long70b": 256}
DECODE_ALL_STEPS = {"tiny", "stuff7b", "mapred7b"}


def f64(t):
    return oracle.bf16_bits_to_f64(bf16_bits(t))


@pytest.fixture(scope="module", params=list(WORKLOADS))
def state(request):
    w = WORKLOADS[request.param]()
    st = bench.setup_stuff(torch, w, torch.device("cuda:0"))
    yield st
    del st
    torch.cuda.empty_cache()


def test_prefill_full_size(orc, state):
    st = state
    w = st["w"]
    bench.run_stuff_step(dict(st, decode_steps=0))
    torch.cuda.synchronize()
    cu, lens = st["cu"], st["lens"]
    print(f"{w.name} prefill: {len(lens)} prompts, {cu[-1]} tokens", flush=True)
    if w.name in PREFILL_FULL:
        # every row and head, in batches of whole prompts
        lse = torch.empty((w.hq, cu[-1]), dtype=torch.float32, device="cuda")
        binding.rag_attn_prefill_varlen(st["q"], st["k"], st["v"], st["o"], lse, st["cu_t"],
                                        st["cu_t"], max(lens), max(lens), w.scale, True)
        torch.cuda.synchronize()
        worst = (0.0, 0.0)
        step = 40
        for s0 in range(0, len(lens), step):
            s1 = min(len(lens), s0 + step)
            a, b = cu[s0], cu[s1]
            lc = [x - a for x in cu[s0:s1 + 1]]
            ro, rl = orc.varlen(f64(st["q"][a:b]), f64(st["k"][a:b]), f64(st["v"][a:b]), lc, lc,
                                w.scale, True)
            mx, mean = G.assert_parity(st["o"][a:b], ro, f"{w.name} prefill seqs {s0}..{s1}")
            worst = (max(worst[0], mx), max(worst[1], mean))
            assert np.max(np.abs(lse[:, a:b].cpu().numpy() - rl)) < 1e-3, "lse"
        print(f"{w.name} prefill full output: max {worst[0]:.3e} mean {worst[1]:.3e}")
        return
    rng = np.random.Generator(np.random.PCG64(7))
    got, want = [], []
    heads_all = list(range(w.hq))
    for s in range(len(lens)):
        L = lens[s]
        k = bf16_bits(st["k"][cu[s]:cu[s + 1]])
        v = bf16_bits(st["v"][cu[s]:cu[s + 1]])
        rows, heads = [], []
        for r in G.sample_rows(L, w.chunk_len, rng, n_random=RANDOM_ROWS[w.name]):
            rows += [r] * w.hq
            heads += heads_all
        o, _ = G.oracle_seq_rows(orc, st["q"][cu[s]:cu[s + 1]], k, v, L, rows, heads, w.scale)
        g = st["o"][cu[s]:cu[s + 1]][torch.as_tensor(rows).long().cuda(),
                                     torch.as_tensor(heads).long().cuda()]
        got.append(g.float().cpu().numpy())
        want.append(o)
    G.assert_parity(np.concatenate(got), np.concatenate(want), f"{w.name} prefill")


def _decode_steps(st):
    w = st["w"]
    n = st["decode_steps"]
    if w.name in DECODE_ALL_STEPS:
        return list(range(n))
    rng = np.random.Generator(np.random.PCG64(19))
    fixed = [0, 1, 127, 255]
    rest = [int(t) for t in rng.choice([t for t in range(n) if t not in fixed], 8, replace=False)]
    return sorted(fixed + rest)


def test_decode_full_size(orc, state):
    st = state
    w = st["w"]
    steps = _decode_steps(st)
    S, n = len(st["lens"]), st["decode_steps"]
    print(f"{w.name} decode: {len(steps)} of {n} steps, {S} sequences", flush=True)
    # run every step in order, as the bench does (pools alternate), keeping outputs
    outs = {}
    pools = st["pools"]
    for t in range(n):
        pool = pools[t % len(pools)]
        binding.rag_attn_decode_paged(st["dq"][t], pool.k_cache, pool.v_cache, st["do"],
                                      pool.block_tables, st["kv_steps"][t], w.scale,
                                      workspace=st["ws"])
        if t in steps:
            outs[t] = st["do"].clone()
    torch.cuda.synchronize()
    heads = list(range(w.hq))
    worst = (0.0, 0.0)
    for p, pool in enumerate(pools):
        ts = [t for t in steps if t % len(pools) == p]
        if not ts:
            continue
        got = torch.stack([outs[t] for t in ts]).float().cpu().numpy()   # [steps, S, hq, d]
        want = np.zeros(got.shape, dtype=np.float64)
        for s, L in enumerate(st["lens"]):
            nk = L + n
            kb, vb = G.dense_kv_of_seq(pool, s, nk)
            k = oracle.bf16_bits_to_f64(kb)
            v = oracle.bf16_bits_to_f64(vb)
            rows = np.repeat(np.asarray(ts, dtype=np.int32), w.hq)
            hs = np.tile(np.asarray(heads, dtype=np.int32), len(ts))
            qr = f64(st["dq"][torch.as_tensor(rows).long().cuda(), s,
                              torch.as_tensor(hs).long().cuda()])
            o, _ = orc.seq_rows(qr, k, v, n, rows, hs, w.hq, w.scale, True)
            want[:, s] = o.reshape(len(ts), w.hq, w.d)
        mx, mean = G.assert_parity(got, want, f"{w.name} decode pool {p} (splits {st['splits']})")
        worst = (max(worst[0], mx), max(worst[1], mean))
    print(f"{w.name} decode: max {worst[0]:.3e} mean {worst[1]:.3e}")


def test_mixed_full_size(orc):
    st = bench.setup_mixed(torch, torch.device("cuda:0"), n_pools=1)
    w = st["w"]
    bench.run_mixed(st, 0)
    torch.cuda.synchronize()
    pool = st["pools"][0]
    rng = np.random.Generator(np.random.PCG64(11))
    heads = list(range(w.hq))
    # every decode row, all heads
    got, want = [], []
    for s in range(st["nd"]):
        n = st["kv"][s]
        k, v = G.dense_kv_of_seq(pool, s, n)
        row = st["cu"][s]
        o, _ = G.oracle_seq_rows(orc, st["q"][row:row + 1], k, v, 1, [0] * w.hq, heads, w.scale)
        got.append(st["o"][row].float().cpu().numpy())
        want.append(o)
    G.assert_parity(np.concatenate(got), np.concatenate(want), "mixed decode rows")
    # chunked-prefill pieces: sampled rows, all heads
    got, want = [], []
    for s in range(st["nd"], len(st["kv"])):
        n, nq = st["kv"][s], st["q_lens"][s]
        k, v = G.dense_kv_of_seq(pool, s, n)
        q0 = st["cu"][s]
        rows, hs = [], []
        for r in G.sample_rows(nq, 512, rng, n_random=1024):
            rows += [r] * w.hq
            hs += heads
        o, _ = G.oracle_seq_rows(orc, st["q"][q0:q0 + nq], k, v, nq, rows, hs, w.scale)
        g = st["o"][q0:q0 + nq][torch.as_tensor(rows).long().cuda(),
                                torch.as_tensor(hs).long().cuda()]
        got.append(g.float().cpu().numpy())
        want.append(o)
    G.assert_parity(np.concatenate(got), np.concatenate(want), "mixed pieces")
