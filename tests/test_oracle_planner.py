"""The oracle's prompt planner against the paper's worked configurations
(tests/golden/planner_examples.json, each case citing its passage)."""
import json
import os

import pytest

from oracle import plan_prompts

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "planner_examples.json")
CASES = json.load(open(GOLDEN))["cases"]


@pytest.mark.parametrize("case", CASES, ids=[f"{c['method']}-{i}" for i, c in enumerate(CASES)])
def test_planner_golden(case):
    cu, dec, owner = plan_prompts(case["method"], case["query_lens"], case["num_chunks"],
                                  case["chunk_len"], case["intermediate_length"],
                                  case["answer_len"])
    lens = [b - a for a, b in zip(cu[:-1], cu[1:])]
    assert lens == case["seq_lens"]
    assert dec == case["decode_lens"]
    assert len(owner) == len(lens) and owner == sorted(owner)


def test_planner_rejects_unknown_method():
    with pytest.raises(ValueError):
        plan_prompts("refine", [1], [1], 1, 1, 1)


def test_planner_empty():
    assert plan_prompts("stuff", [], [], 512, 0, 0) == ([0], [], [])
