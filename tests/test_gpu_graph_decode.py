"""The decode steps replayed from a HIP graph, as bench.py times them: every
replay, with eager launches and synchronisations of the program in between,
gives the eager launches' last output bit for bit, the split-merge counters
stay usable by eager calls after the replays, and the last step matches the
fp64 oracle.  Three prompts x 8 kv heads leave CUs idle, so the default policy
runs balanced decode units whose split partials merge in the kernel."""
import os
import sys

import pytest
import torch

import gpu_support as G
from paper_2412_10543_amd.workloads import Workload

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402

pytestmark = pytest.mark.gpu


def test_decode_graph_replays_match_eager(orc):
    w = Workload("graph-check", "stuff", [40, 64, 17], [5, 9, 2], 512, 0, 8, 32, 8, 128,
                 seed=1400)
    dev = torch.device("cuda:0")
    st = bench.setup_stuff(torch, w, dev)
    assert st["decode_steps"] == 8
    bench.run_stuff_step(st, None, plan=False)
    torch.cuda.synchronize()
    bench.capture_decode(torch, st)                      # captures, checks one replay
    for i in range(3):
        print(f"graph replay {i}", flush=True)
        bench.run_stuff_step(st, None, plan=False, decode=False)   # eager prefill between
        torch.cuda.synchronize()
        bench.check_decode_replay(torch, st)             # zero, replay, compare bitwise
    st["do"].zero_()
    bench.run_decode_launches(st)
    torch.cuda.synchronize()
    assert torch.equal(st["do"].view(torch.int16), st["do_eager"].view(torch.int16)), \
        "eager launches after the replays"
    t = st["decode_steps"] - 1
    pool = st["pools"][t % len(st["pools"])]
    ref = G.oracle_paged(orc, st["dq"][t], pool, w.scale,
                         kv_lens=[int(x) for x in st["kv_steps"][t].cpu()])
    G.assert_parity(st["do"], ref, "last decode step")
