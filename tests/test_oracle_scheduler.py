"""Pins of the oracle's configuration pruning and memory-aware choice
(oracle/scheduler.py), on the CPU: the paper's worked mapping examples,
best-fit example and scheduling illustration with memory requirements worked
out by hand (tests/golden/scheduler_examples.json), its stated fallback rules,
properties every choice must have, and planted mistakes that the pins catch."""
import importlib.util
import json
import os

import numpy as np
import pytest

from oracle import scheduler as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "scheduler_examples.json")
G = json.load(open(GOLDEN))
SHAPE = dict(query_len=64, chunk_len=512, answer_len=32, bytes_per_token=131072)


def _profile(p):
    return dict(p, summary_range=tuple(p["summary_range"]))


@pytest.mark.parametrize("case", G["mapping"], ids=lambda c: c["cite"][:40])
def test_paper_mapping_examples(case):
    methods, chunks, ils = S.prune(case["profile"]["complexity_high"],
                                   case["profile"]["joint_reasoning"],
                                   case["profile"]["pieces"],
                                   tuple(case["profile"]["summary_range"]))
    assert list(methods) == case["methods"]
    assert list(chunks) == case["num_chunks"] and list(ils) == case["intermediate_length"]


def test_paper_best_fit_example():
    b = G["best_fit"]
    shape = b["shape"]
    n_fit = b["fits_chunks"]
    # memory between what n_fit and n_fit + 1 stuff chunks need
    lo = S.kv_bytes(n_fit * shape["chunk_len"] + shape["query_len"] + shape["answer_len"],
                    shape["bytes_per_token"])
    hi = S.kv_bytes((n_fit + 1) * shape["chunk_len"] + shape["query_len"] + shape["answer_len"],
                    shape["bytes_per_token"])
    for avail in (lo, (lo + hi) // 2, hi - 1):
        got = S.choose(_profile(b["profile"]), shape, avail)
        assert {k: got[k] for k in b["choice"]} == b["choice"]


@pytest.mark.parametrize("case", G["requirements"], ids=lambda c: c["method"])
def test_hand_computed_requirements(case):
    shape = {k: v for k, v in G["shape_7b"].items() if not k.startswith("_")}
    assert S.requirement(case["method"], case["num_chunks"], case["intermediate_length"],
                         shape) == case["kv_bytes"]
    assert S.kv_bytes(case["tokens"], shape["bytes_per_token"]) == case["kv_bytes"]


@pytest.mark.parametrize("case", G["scheduling"]["cases"], ids=lambda c: str(c["available"]))
def test_scheduling_illustration(case):
    shape = {k: v for k, v in G["shape_7b"].items() if not k.startswith("_")}
    got = S.choose(_profile(G["scheduling"]["profile"]), shape, case["available"])
    assert got == case["choice"]


@pytest.mark.parametrize("case", G["fallback"]["cases"], ids=lambda c: c["choice"]["method"])
def test_fallback_examples(case):
    shape = {k: v for k, v in G["shape_7b"].items() if not k.startswith("_")}
    assert S.choose(_profile(case["profile"]), shape, case["available"]) == case["choice"]


def test_illustration_map_reduce_starts_where_stuff_queues():
    """With 20 chunks and intermediate length 100, map_reduce needs less free
    memory to start than stuff, so some memory levels admit it and not stuff."""
    shape = {k: v for k, v in G["shape_7b"].items() if not k.startswith("_")}
    stuff = S.requirement(S.STUFF, 20, 0, shape)
    mr = S.requirement(S.MAP_REDUCE, 20, 100, shape)
    assert mr < stuff
    assert S.fits(S.MAP_REDUCE, 20, 100, shape, stuff - 1)
    assert not S.fits(S.STUFF, 20, 0, shape, stuff - 1)


def test_two_percent_buffer():
    # 1000 tokens of 100 bytes: 100,000 bytes plus 2%
    assert S.kv_bytes(1000, 100) == 102000
    assert S.kv_bytes(1, 1) == 2     # rounded up to a whole byte


def test_fallback_rules():
    """None of the pruned space fits: joint reasoning -> stuff, otherwise
    map_rerank, with as many chunks as fit; nothing fits -> wait."""
    # high complexity: map_reduce's mappers start as memory allows, so it is
    # chosen as long as its largest call fits -- here a mapper of 512 + 64 + 30
    # tokens fits where 2 stuff chunks do, and the reduce call of 12 summaries
    joint = dict(complexity_high=True, joint_reasoning=True, pieces=4, summary_range=(30, 200))
    two = S.kv_bytes(2 * 512 + 64 + 32, SHAPE["bytes_per_token"])
    got = S.choose(joint, SHAPE, two)
    assert got["method"] == "map_reduce" and not got["fallback"]
    no_joint = dict(complexity_high=False, joint_reasoning=False, pieces=5, summary_range=(30, 200))
    one_call = S.kv_bytes(512 + 64 + 32, SHAPE["bytes_per_token"])
    # three answer calls fit, the pruned minimum of five does not
    got = S.choose(no_joint, SHAPE, S.kv_bytes(3 * (512 + 64 + 32), SHAPE["bytes_per_token"]))
    assert got == dict(method="map_rerank", num_chunks=3, intermediate_length=0,
                       kv_bytes=S.kv_bytes(3 * (512 + 64 + 32), SHAPE["bytes_per_token"]),
                       fallback=True)
    assert S.choose(no_joint, SHAPE, one_call - 1) is None


def test_stuff_fallback_counts_chunks():
    low = dict(complexity_high=False, joint_reasoning=True, pieces=6, summary_range=(30, 200))
    for k in (1, 2, 5):
        avail = S.kv_bytes(k * 512 + 64 + 32, SHAPE["bytes_per_token"])
        got = S.choose(low, SHAPE, avail)
        assert got["method"] == "stuff" and got["num_chunks"] == k and got["fallback"]


def test_choice_properties():
    """Every choice fits, lies in the pruned space unless it is a fallback,
    and no fitting configuration of the space needs more memory; more memory
    never yields a smaller requirement."""
    rng = np.random.Generator(np.random.PCG64(3))
    for _ in range(60):
        p = dict(complexity_high=bool(rng.integers(2)), joint_reasoning=bool(rng.integers(2)),
                 pieces=int(rng.integers(1, 11)), summary_range=(30, int(rng.integers(30, 201))))
        methods, chunks, ils = S.prune(p["complexity_high"], p["joint_reasoning"], p["pieces"],
                                       p["summary_range"])
        prev = -1
        for avail in sorted(int(x) for x in rng.integers(1 << 20, 8 << 30, size=6)):
            got = S.choose(p, SHAPE, avail)
            if got is None:
                assert prev == -1
                continue
            assert S.fits(got["method"], got["num_chunks"], got["intermediate_length"], SHAPE, avail)
            if not got["fallback"]:
                assert got["method"] in methods and chunks[0] <= got["num_chunks"] <= chunks[1]
                for m, n, il in S.candidates(methods, chunks, ils):
                    if S.fits(m, n, il, SHAPE, avail):
                        assert S.requirement(m, n, il, SHAPE) <= got["kv_bytes"]
            assert got["kv_bytes"] >= prev or got["fallback"]
            prev = got["kv_bytes"] if not got["fallback"] else prev


# Planted mistakes, each a plausible misreading or slip in oracle/scheduler.py:
# (name, original text, planted text).
SRC = open(S.__file__).read()
MUTANTS = [
    ("all_mappers_together", "return [[chunk_len + query_len + il], [n * il + query_len + answer_len]]",
     "return [[chunk_len + query_len + il] * n, [n * il + query_len + answer_len]]"),
    ("reduce_without_answer", "[n * il + query_len + answer_len]]", "[n * il + query_len]]"),
    ("mapper_without_summary", "return [[chunk_len + query_len + il], [n",
     "return [[chunk_len + query_len], [n"),
    ("rerank_one_call", "return [[chunk_len + query_len + answer_len] * n]",
     "return [[chunk_len + query_len + answer_len]]"),
    ("stuff_without_query", "return [[n * chunk_len + query_len + answer_len]]",
     "return [[n * chunk_len + answer_len]]"),
    ("buffer_20_percent", "* 102 // 100", "* 120 // 100"),
    ("lowest_requirement", "if best_key is None or key > best_key:",
     "if best_key is None or key < best_key:"),
    ("fallback_method_swapped", "m = STUFF if profile[\"joint_reasoning\"] else MAP_RERANK",
     "m = MAP_RERANK if profile[\"joint_reasoning\"] else STUFF"),
    ("fallback_fewest_chunks", "for n in range(chunks[1], 0, -1):", "for n in range(1, chunks[1] + 1):"),
    ("complexity_ignored", "elif not complexity_high:", "elif False:"),
]


def _pins(mod):
    """The golden pins above, run against a module; returns the failures."""
    shape = {k: v for k, v in G["shape_7b"].items() if not k.startswith("_")}
    failed = []
    for c in G["requirements"]:
        if mod.requirement(c["method"], c["num_chunks"], c["intermediate_length"],
                           shape) != c["kv_bytes"]:
            failed.append(("requirement", c["method"]))
    for c in G["scheduling"]["cases"]:
        if mod.choose(_profile(G["scheduling"]["profile"]), shape, c["available"]) != c["choice"]:
            failed.append(("scheduling", c["available"]))
    for c in G["fallback"]["cases"]:
        if mod.choose(_profile(c["profile"]), shape, c["available"]) != c["choice"]:
            failed.append(("fallback", c["available"]))
    for c in G["mapping"]:
        p = c["profile"]
        m, ch, il = mod.prune(p["complexity_high"], p["joint_reasoning"], p["pieces"],
                              tuple(p["summary_range"]))
        if list(m) != c["methods"] or list(ch) != c["num_chunks"]:
            failed.append(("mapping", c["cite"][:20]))
    return failed


def _load(tmp_path, name, src):
    f = tmp_path / f"sched_{name}.py"
    f.write_text(src)
    spec = importlib.util.spec_from_file_location(f"sched_{name}", str(f))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_scheduler_mutant_is_caught(tmp_path, name, old, new):
    assert SRC.count(old) == 1, f"mutation site for {name} not found once"
    assert _pins(_load(tmp_path, name, SRC.replace(old, new))), \
        f"no pin catches the planted mistake {name}"


def test_scheduler_unmodified_copy_passes(tmp_path):
    assert _pins(_load(tmp_path, "clean", SRC)) == []
