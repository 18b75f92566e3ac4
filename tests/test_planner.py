"""The library's configuration planner (rag_prune_config_space,
rag_config_kv_bytes, rag_choose_config) against the oracle's
(oracle/scheduler.py) on the CPU: identical decisions over random profiles,
request shapes and memory levels, the paper's worked examples, and argument
validation.  rag_device_free_memory is checked on the GPU."""
import json
import os

import numpy as np
import pytest

from oracle import scheduler as S
from paper_2412_10543_amd import binding

pytestmark = pytest.mark.skipif(not os.path.exists(binding.LIBRARY),
                                reason="librag_attn.so not built")
GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "scheduler_examples.json")))


def test_prune_matches_oracle_and_paper():
    for case in GOLDEN["mapping"]:
        p = case["profile"]
        got = binding.rag_prune_config_space(p["complexity_high"], p["joint_reasoning"],
                                             p["pieces"], p["summary_range"])
        assert list(got[0]) == case["methods"]
        assert list(got[1]) == case["num_chunks"] and list(got[2]) == case["intermediate_length"]
    for ch in (0, 1):
        for jr in (0, 1):
            for n in (1, 3, 10):
                want = S.prune(bool(ch), bool(jr), n, (30, 200))
                assert binding.rag_prune_config_space(ch, jr, n, (30, 200)) == want


def test_kv_bytes_matches_oracle():
    rng = np.random.Generator(np.random.PCG64(1))
    for _ in range(300):
        m = ["stuff", "map_reduce", "map_rerank"][int(rng.integers(3))]
        n, il = int(rng.integers(0, 40)), int(rng.integers(0, 400))
        shape = dict(query_len=int(rng.integers(0, 300)), chunk_len=int(rng.integers(0, 2048)),
                     answer_len=int(rng.integers(0, 128)),
                     bytes_per_token=int(rng.integers(1, 1 << 19)))
        got = binding.rag_config_kv_bytes(m, n, il if m == "map_reduce" else 0,
                                          shape["query_len"], shape["chunk_len"],
                                          shape["answer_len"], shape["bytes_per_token"])
        assert got == S.requirement(m, n, il if m == "map_reduce" else 0, shape)


def test_choose_matches_oracle():
    rng = np.random.Generator(np.random.PCG64(2))
    for trial in range(250):
        p = dict(complexity_high=bool(rng.integers(2)), joint_reasoning=bool(rng.integers(2)),
                 pieces=int(rng.integers(1, 11)))
        lo = int(rng.integers(20, 120))
        p["summary_range"] = (lo, lo + int(rng.integers(0, 90)))
        shape = dict(query_len=int(rng.integers(8, 200)), chunk_len=int(rng.choice([256, 512, 1024])),
                     answer_len=int(rng.integers(1, 64)),
                     bytes_per_token=int(rng.choice([65536, 131072, 163840])))
        # memory levels from "nothing fits" to "everything fits"
        avail = int(np.exp(rng.uniform(np.log(1 << 16), np.log(64 << 30))))
        want = S.choose(p, shape, avail)
        got = binding.rag_choose_config(p["complexity_high"], p["joint_reasoning"], p["pieces"],
                                        p["summary_range"], shape["query_len"],
                                        shape["chunk_len"], shape["answer_len"],
                                        shape["bytes_per_token"], avail)
        assert got == want, (trial, p, shape, avail)


def test_best_fit_example_through_library():
    b = GOLDEN["best_fit"]
    sh = b["shape"]
    lo = S.kv_bytes(b["fits_chunks"] * sh["chunk_len"] + sh["query_len"] + sh["answer_len"],
                    sh["bytes_per_token"])
    got = binding.rag_choose_config(b["profile"]["complexity_high"], b["profile"]["joint_reasoning"],
                                    b["profile"]["pieces"], b["profile"]["summary_range"],
                                    sh["query_len"], sh["chunk_len"], sh["answer_len"],
                                    sh["bytes_per_token"], lo)
    assert {k: got[k] for k in b["choice"]} == b["choice"]


def _choose(profile, shape, avail):
    return binding.rag_choose_config(profile["complexity_high"], profile["joint_reasoning"],
                                     profile["pieces"], tuple(profile["summary_range"]),
                                     shape["query_len"], shape["chunk_len"], shape["answer_len"],
                                     shape["bytes_per_token"], avail)


def test_hand_computed_requirements_through_library():
    sh = GOLDEN["shape_7b"]
    for c in GOLDEN["requirements"]:
        assert binding.rag_config_kv_bytes(c["method"], c["num_chunks"], c["intermediate_length"],
                                           sh["query_len"], sh["chunk_len"], sh["answer_len"],
                                           sh["bytes_per_token"]) == c["kv_bytes"], c["cite"]


def test_scheduling_and_fallback_examples_through_library():
    """A complex profile: ample memory gives stuff, memory below stuff's
    minimum but above one map_reduce call gives map_reduce, then the stuff
    fallback, then a wait; and the two fallback methods."""
    sh = GOLDEN["shape_7b"]
    for c in GOLDEN["scheduling"]["cases"]:
        assert _choose(GOLDEN["scheduling"]["profile"], sh, c["available"]) == c["choice"], c["why"]
    for c in GOLDEN["fallback"]["cases"]:
        assert _choose(c["profile"], sh, c["available"]) == c["choice"], c["why"]


@pytest.mark.parametrize("args", [
    dict(pieces=0), dict(summary_range=(50, 40)), dict(summary_range=(0, 10)),
    dict(complexity_high=2), dict(bytes_per_token=0), dict(query_len=-1),
    dict(available=-5)])
def test_choose_validation(args):
    a = dict(complexity_high=1, joint_reasoning=1, pieces=3, summary_range=(30, 200), query_len=64,
             chunk_len=512, answer_len=32, bytes_per_token=131072, available=1 << 30)
    a.update(args)
    L = binding.lib()
    prof = binding.QueryProfile(a["complexity_high"], a["joint_reasoning"], a["pieces"],
                                a["summary_range"][0], a["summary_range"][1])
    shape = binding.RequestShape(a["query_len"], a["chunk_len"], a["answer_len"],
                                 a["bytes_per_token"])
    out = binding.Config()
    import ctypes
    st = L.rag_choose_config(ctypes.byref(prof), ctypes.byref(shape), a["available"],
                             ctypes.byref(out))
    assert st == binding.RAG_ERR_INVALID_ARG
    assert binding.rag_last_error().startswith("planner")


def test_no_fit_status():
    assert binding.rag_choose_config(0, 0, 2, (30, 60), 64, 1024, 16, 131072, 1000) is None


@pytest.mark.gpu
def test_device_free_memory():
    free, total = binding.rag_device_free_memory()
    assert 0 < free <= total and total > (100 << 30)    # an MI355X has 288 GB
