"""A synthetic query stream through the planner and the kernels
(paper_2412_10543_amd/stream.py): every query completes, every configuration
the engine ran is the one the oracle planner chooses for the memory free at
its admission, memory and pages are all returned at the end."""
import pytest
import torch

from oracle import scheduler as S
from paper_2412_10543_amd import stream

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("budget_gb,n,rate", [(1, 10, 400.0), (4, 16, 200.0)])
def test_stream_completes(budget_gb, n, rate):
    eng = stream.Engine(kv_budget_bytes=int(budget_gb * (1 << 30)), chunk_len=256, answer_len=8,
                        layers=32, seed=3)
    queries = stream.synthetic_queries(n, rate, seed=n)
    seen = []
    orig_choose = stream.binding.rag_choose_config

    def spy(*args):
        got = orig_choose(*args)
        seen.append((args, got))
        return got
    stream.binding.rag_choose_config = spy
    try:
        res = stream.run_stream(queries, eng)
    finally:
        stream.binding.rag_choose_config = orig_choose
    assert res["completed"] == n, res
    assert eng.used == 0 and sorted(eng.free_blocks) == list(range(eng.num_blocks))
    assert res["prefill_launches"] > 0 and res["decode_launches"] > 0
    for args, got in seen:
        ch, jr, pieces, rng_, ql, cl, al, bpt, avail = args
        want = S.choose(dict(complexity_high=ch, joint_reasoning=jr, pieces=pieces,
                             summary_range=tuple(rng_)),
                        dict(query_len=ql, chunk_len=cl, answer_len=al, bytes_per_token=bpt), avail)
        assert got == want
    torch.cuda.synchronize()
