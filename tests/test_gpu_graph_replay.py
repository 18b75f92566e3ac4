"""Launches captured in a HIP graph and replayed, as a serving loop would run
them: the packed prefill (several query tiles per workgroup, LSE), the mixed
decode + chunked-prefill launch with split-KV merges, and the int4 GEMM split
over the weight groups.  Every replay, with eager launches of other inputs and
synchronisations in between, gives the eager result bit for bit; the split
counters in the workspaces stay usable by eager calls after the replays; the
outputs match the fp64 oracle.  The same three calls enqueued on three streams
at once (each with its own workspace) give the results computed alone."""
import numpy as np
import pytest
import torch

import gpu_support as G
import oracle
from paper_2412_10543_amd import binding
from paper_2412_10543_amd.workloads import awq_problem, normal_bf16, paged_pool

pytestmark = pytest.mark.gpu


def _capture(fn, calls=1):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            for _ in range(calls):
                fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    return g


def _same(a, b):
    if a.dtype == torch.bfloat16:
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_prefill_graph_replays(orc):
    lq = [576, 130, 1, 700, 64]
    hq, hkv, d = 32, 8, 128
    sc = G.scale_for(d)
    q, k, v = G.prefill_inputs(lq, lq, hq, hkv, d, seed=1500)
    q2, k2, v2 = G.prefill_inputs(lq, lq, hq, hkv, d, seed=1510)
    cu = G.to_dev_i32(G.cu_from_lens(lq))
    o = torch.empty_like(q)
    lse = torch.empty((hq, q.shape[0]), dtype=torch.float32, device="cuda")
    o2, lse2 = torch.empty_like(o), torch.empty_like(lse)

    def call(qq, kk, vv, oo, ll):
        binding.rag_attn_prefill_varlen(qq, kk, vv, oo, ll, cu, cu, max(lq), max(lq), sc, True)

    with G.env("RAG_ATTN_PF_ITEMS", 3):
        call(q, k, v, o, lse)
        torch.cuda.synchronize()
        want_o, want_l = o.clone(), lse.clone()
        g = _capture(lambda: call(q, k, v, o, lse))
        for i in range(3):
            print(f"prefill graph replay {i}", flush=True)
            call(q2, k2, v2, o2, lse2)                   # eager work on other buffers
            torch.cuda.synchronize()
            o.zero_()
            lse.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert _same(o, want_o) and _same(lse, want_l), f"replay {i}"
    ro, rl = G.oracle_prefill(orc, q, k, v, lq, lq, sc)
    G.assert_parity(o, ro, "prefill after replays")
    fin = np.isfinite(rl)
    got_l = lse.cpu().numpy().astype(np.float64)
    assert np.max(np.abs(got_l[fin] - rl[fin])) <= 1e-3


def test_mixed_split_graph_replays(orc):
    hq, hkv, d = 32, 8, 128
    sc = G.scale_for(d)
    dec_kv = [2000, 17, 3000, 900, 1]
    pieces = [(300, 500), (129, 129)]
    kv = dec_kv + [nq + p for nq, p in pieces]
    pool = paged_pool(kv, hkv, d, 1520, device="cuda")
    q_lens = [1] * len(dec_kv) + [nq for nq, _ in pieces]
    cu_l = G.cu_from_lens(q_lens)
    cu, kl = G.to_dev_i32(cu_l), G.to_dev_i32(pool.kv_lens)
    q = normal_bf16((cu_l[-1], hq, d), 1521, "cuda")
    q2 = normal_bf16((cu_l[-1], hq, d), 1522, "cuda")
    o, o2 = torch.empty_like(q), torch.empty_like(q)
    nd, splits = len(dec_kv), 4
    ws = G.workspace_for(nd, hq, hkv, d, pool.block_tables.shape[1], splits)
    assert ws is not None

    def call(qq, oo):
        binding.rag_attn_decode_paged(qq, pool.k_cache, pool.v_cache, oo, pool.block_tables, kl,
                                      sc, cu_seqlens_q=cu, num_decode_seqs=nd,
                                      max_seqlen_q=max(q_lens), num_splits=splits, workspace=ws)

    call(q, o)
    torch.cuda.synchronize()
    want = o.clone()
    g = _capture(lambda: call(q, o))
    for i in range(3):
        print(f"mixed graph replay {i}", flush=True)
        call(q2, o2)                                     # eager call on the same workspace
        torch.cuda.synchronize()
        o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert _same(o, want), f"replay {i}"
    o2b = torch.empty_like(o2)
    call(q2, o2b)                                        # eager after the replays
    torch.cuda.synchronize()
    assert _same(o2b, o2)
    G.assert_parity(o, G.oracle_paged(orc, q, pool, sc, cu_q=cu_l), "mixed after replays")


def test_awq_split_graph_replays():
    M, N, K = 16, 1024, 14336
    p = awq_problem(M, N, K, seed=1530, device="cuda")
    p2 = awq_problem(M, N, K, seed=1531, device="cuda")
    qw = torch.from_numpy(binding.rag_awq_pack_weights(p.codes)).cuda()
    sc, z = p.scales.cuda(), torch.from_numpy(p.zeros).cuda()
    n = binding.rag_awq_workspace_size(M, N, K)
    assert n > 0, "this shape splits the groups"
    ws = torch.zeros(n, dtype=torch.uint8, device="cuda")
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    y2 = torch.empty_like(y)
    binding.rag_awq_gemm(p.x, qw, sc, z, y, ws)
    torch.cuda.synchronize()
    want = y.clone()
    g = _capture(lambda: binding.rag_awq_gemm(p.x, qw, sc, z, y, ws), calls=3)
    for i in range(3):
        print(f"awq graph replay {i}", flush=True)
        binding.rag_awq_gemm(p2.x, qw, sc, z, y2, ws)   # eager call on the same workspace
        torch.cuda.synchronize()
        y.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert _same(y, want), f"replay {i}"
    assert int(ws[:4 * (N // 128)].count_nonzero()) == 0   # arrival counters reset
    x = p.x.float().cpu().numpy().astype(np.float64)
    ref = oracle.awq_gemm(x, p.codes, p.zeros, p.scales.float().numpy().astype(np.float64), 128)
    G.assert_parity(y.float().cpu().numpy().astype(np.float64), ref, "awq after replays")


def test_concurrent_streams_match_sequential():
    """A prefill, a split-KV decode (own workspace) and a split int4 GEMM (own
    workspace) enqueued on three streams so that they may run at the same
    time, four rounds: every result equals the one computed alone."""
    hq, hkv, d = 32, 8, 128
    sc = G.scale_for(d)
    lq = [576, 300, 1000]
    q, k, v = G.prefill_inputs(lq, lq, hq, hkv, d, seed=1540)
    cu = G.to_dev_i32(G.cu_from_lens(lq))
    kv = [3000, 17, 900, 4000]
    pool = paged_pool(kv, hkv, d, 1541, device="cuda")
    kl = G.to_dev_i32(pool.kv_lens)
    dq = normal_bf16((len(kv), hq, d), 1542, "cuda")
    ws_d = G.workspace_for(len(kv), hq, hkv, d, pool.block_tables.shape[1], 4)
    M, N, K = 16, 1024, 14336
    p = awq_problem(M, N, K, seed=1543, device="cuda")
    qw = torch.from_numpy(binding.rag_awq_pack_weights(p.codes)).cuda()
    asc, az = p.scales.cuda(), torch.from_numpy(p.zeros).cuda()
    ws_a = torch.zeros(binding.rag_awq_workspace_size(M, N, K), dtype=torch.uint8, device="cuda")

    def prefill(o, stream):
        binding.rag_attn_prefill_varlen(q, k, v, o, None, cu, cu, max(lq), max(lq), sc, True,
                                        stream=stream)

    def decode(o, stream):
        binding.rag_attn_decode_paged(dq, pool.k_cache, pool.v_cache, o, pool.block_tables, kl,
                                      sc, num_splits=4, workspace=ws_d, stream=stream)

    def gemm(y, stream):
        binding.rag_awq_gemm(p.x, qw, asc, az, y, ws_a, stream=stream)

    alone = [torch.empty_like(q), torch.empty_like(dq),
             torch.empty((M, N), dtype=torch.bfloat16, device="cuda")]
    for fn, out in zip((prefill, decode, gemm), alone):
        fn(out, None)
        torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(3)]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for r in range(4):
        print(f"concurrent round {r}", flush=True)
        outs = [torch.empty_like(a) for a in alone]
        torch.cuda.synchronize()
        for fn, out, s in zip((prefill, decode, gemm), outs, streams):
            with torch.cuda.stream(s):
                fn(out, s.cuda_stream)
        torch.cuda.synchronize()
        for a, b in zip(alone, outs):
            assert _same(a, b), f"round {r}"
