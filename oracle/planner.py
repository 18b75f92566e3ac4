"""Prompt assembly for each synthesis method, written straight from the
method definitions: the oracle's side of the packed-batch descriptor.

Test infrastructure only (see ``oracle/__init__.py``).

Sec. "RAG systems and configurations" defines the three synthesis methods and
the knobs num_chunks and intermediate_length:
  * stuff: every retrieved chunk and the query go into one prompt; the LLM
    answers in one call;
  * map_reduce: one mapper call per chunk (chunk + query) produces a summary of
    intermediate_length tokens; a reduce call reads the summaries and the query;
  * map_rerank: one call per chunk (chunk + query), each producing an answer;
    the answer with the highest confidence is kept.
Readings used (the paper gives no template): chunks come first in retrieval
order, then the query; no template tokens; intermediate_length and the answer
length are counted in tokens.
"""
from __future__ import annotations

STUFF = "stuff"
MAP_REDUCE_MAP = "map_reduce_map"
MAP_REDUCE_REDUCE = "map_reduce_reduce"
MAP_RERANK = "map_rerank"
METHODS = (STUFF, MAP_REDUCE_MAP, MAP_REDUCE_REDUCE, MAP_RERANK)


def plan_prompts(method, query_lens, num_chunks, chunk_len,
                 intermediate_length, answer_len):
    """Return (cu_seqlens, decode_lens, owner) for a list of queries.

    cu_seqlens has one more entry than there are LLM calls; decode_lens[i] is
    how many tokens call i generates; owner[i] is the index of the query that
    issued it.
    """
    if method not in METHODS:
        raise ValueError(f"unknown synthesis method {method!r}")
    lens, dec, owner = [], [], []
    for qi, (lq, n) in enumerate(zip(query_lens, num_chunks)):
        if method == STUFF:
            # one prompt: n chunks then the query
            lens.append(n * chunk_len + lq)
            dec.append(answer_len)
            owner.append(qi)
        elif method == MAP_REDUCE_MAP:
            # n mapper prompts: one chunk then the query; each writes a summary
            for _ in range(n):
                lens.append(chunk_len + lq)
                dec.append(intermediate_length)
                owner.append(qi)
        elif method == MAP_REDUCE_REDUCE:
            # one prompt: the n summaries then the query
            lens.append(n * intermediate_length + lq)
            dec.append(answer_len)
            owner.append(qi)
        else:  # MAP_RERANK
            # n independent prompts, one per chunk, each answering the query
            for _ in range(n):
                lens.append(chunk_len + lq)
                dec.append(answer_len)
                owner.append(qi)
    cu = [0]
    for length in lens:
        cu.append(cu[-1] + length)
    return cu, dec, owner
