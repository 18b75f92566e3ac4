"""Configuration pruning and memory-aware choice, written from the paper's
text: the oracle's side of the host planner.

Test infrastructure only (see ``oracle/__init__.py``).

Sec. "Mapping query profiles to RAG configurations", Algorithm 1 (rule-based
mapping): from the profile (query complexity High/Low, joint reasoning
Yes/No, pieces of information n, summarization length range) --
  * no joint reasoning            -> map_rerank;
  * joint reasoning, low complexity -> stuff;
  * joint reasoning, high complexity -> stuff or map_reduce;
  * num_chunks in [n, 3n]; intermediate_length in the summary-length range.

Sec. "Joint configuration-scheduling adaptation": the memory requirement of a
configuration follows from its token counts and the model's bytes per token,
plus a 2% buffer; it is compared with the available GPU memory to see what
fits, and among the configurations of the pruned space that fit, the one with
the highest requirement is chosen; if none fits, a cheaper configuration just
outside the space is used -- map_rerank (no joint reasoning) or stuff (joint
reasoning) with as many chunks as fit -- and if not even that fits, the
request waits.

Readings (the paper gives no formulas):
  * a call's KV holds its prompt and the tokens it generates (answer_len for
    an answer, intermediate_length for a mapper's summary);
  * the requirement is ONE quantity, used both to decide fit and to rank: the
    KV memory the configuration must have free to start.  stuff: its one call
    of n*C + Lq prompt tokens.  map_rerank: its n calls of C + Lq, which run
    together (the fallback takes "as many chunks as fit").  map_reduce: its
    largest single call -- a mapper (C + Lq + IL) or the reduce call
    (n*IL + Lq + answer) -- because its mappers enter the running batch one by
    one as memory allows and the reduce call runs after they have finished
    (the scheduling illustration: with 20 chunks and intermediate length 100,
    map_reduce starts in memory where stuff has to queue, so its requirement
    is below stuff's);
  * ties go to more chunks, then a longer intermediate length, then the method
    listed first (stuff, map_reduce, map_rerank).
"""
from __future__ import annotations

STUFF, MAP_REDUCE, MAP_RERANK = "stuff", "map_reduce", "map_rerank"
METHOD_ORDER = (STUFF, MAP_REDUCE, MAP_RERANK)


def prune(complexity_high: bool, joint_reasoning: bool, pieces: int, summary_range):
    """Algorithm 1: (methods, (chunks_min, chunks_max), (il_min, il_max))."""
    if not joint_reasoning:
        methods = (MAP_RERANK,)
    elif not complexity_high:
        methods = (STUFF,)
    else:
        methods = (STUFF, MAP_REDUCE)
    return methods, (pieces, 3 * pieces), (summary_range[0], summary_range[1])


def kv_bytes(tokens: int, bytes_per_token: int) -> int:
    """KV memory of `tokens` tokens with the 2% buffer, rounded up to a byte."""
    return -(-tokens * bytes_per_token * 102 // 100)


def resident_sets(method, n, il, query_len, chunk_len, answer_len):
    """Token counts of the groups of calls that must be resident together for
    the configuration to run: one group per start condition."""
    if method == STUFF:
        return [[n * chunk_len + query_len + answer_len]]
    if method == MAP_RERANK:
        return [[chunk_len + query_len + answer_len] * n]
    # map_reduce: any one mapper (the rest follow as memory frees), then the
    # reduce call once the mappers are done
    return [[chunk_len + query_len + il], [n * il + query_len + answer_len]]


def requirement(method, n, il, shape):
    """Memory the configuration needs free to start (see the readings)."""
    sets = resident_sets(method, n, il, shape["query_len"], shape["chunk_len"],
                         shape["answer_len"])
    return max(kv_bytes(sum(s), shape["bytes_per_token"]) for s in sets)


def fits(method, n, il, shape, available: int) -> bool:
    return requirement(method, n, il, shape) <= available


def candidates(methods, chunks, ils):
    for m in methods:
        for n in range(chunks[0], chunks[1] + 1):
            if m == MAP_REDUCE:
                for il in range(ils[0], ils[1] + 1):
                    yield m, n, il
            else:
                yield m, n, 0


def choose(profile, shape, available: int):
    """Returns dict(method, num_chunks, intermediate_length, kv_bytes,
    fallback) or None when nothing fits (the request waits)."""
    methods, chunks, ils = prune(profile["complexity_high"], profile["joint_reasoning"],
                                 profile["pieces"], profile["summary_range"])
    best, best_key = None, None
    for m, n, il in candidates(methods, chunks, ils):
        if not fits(m, n, il, shape, available):
            continue
        key = (requirement(m, n, il, shape), n, il, -METHOD_ORDER.index(m))
        if best_key is None or key > best_key:
            best, best_key = (m, n, il), key
    if best is not None:
        m, n, il = best
        return dict(method=m, num_chunks=n, intermediate_length=il,
                    kv_bytes=requirement(m, n, il, shape), fallback=False)
    # nothing in the pruned space fits: a cheaper fixed method, as many chunks as fit
    m = STUFF if profile["joint_reasoning"] else MAP_RERANK
    for n in range(chunks[1], 0, -1):
        if fits(m, n, 0, shape, available):
            return dict(method=m, num_chunks=n, intermediate_length=0,
                        kv_bytes=requirement(m, n, 0, shape), fallback=True)
    return None
