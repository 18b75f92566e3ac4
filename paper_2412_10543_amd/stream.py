"""A synthetic stream of RAG queries driven through the configuration planner
and the attention kernels: a small continuous-batching loop over the C ABI.

Each query arrives (Poisson arrivals, as in the paper's evaluation, Sec.
"Setup") with a profile; when the engine admits it, rag_choose_config picks its
configuration from the KV memory free at that moment (Sec. "Joint
configuration-scheduling adaptation"), and the configuration becomes LLM calls
whose prompt and decode lengths come from rag_plan_prompts (one stuff call, n
mappers then a reduce call, or n map_rerank calls).  An engine iteration
  1. admits waiting queries in arrival order while the planner finds a
     configuration that fits (a query that does not fit waits, and so do the
     queries behind it), and admits queued calls (mappers, reduce calls) whose
     KV fits;
  2. prefills the prompts of the newly admitted calls in one packed varlen
     launch and writes their K/V into the paged cache (rag_kv_cache_write);
  3. runs one decode step for every running call: the new token's K/V is
     written into its page, then one paged decode launch;
  4. retires calls that have generated their tokens and frees their pages; a
     map_reduce query's reduce call is queued once all its mappers are done.
The clock advances by the measured GPU time of each iteration.  The attention
is one transformer layer's (the kernels' unit of work); the memory the planner
sees is the whole model's KV (bytes per token over all layers), and the paged
pool holds the same number of tokens.  Q, K and V values are seeded random
data (only shapes and timing matter here).

Orchestration only: every attention, KV write and prompt plan runs in the
library.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np
import torch

from . import binding

BLOCK = 16


@dataclasses.dataclass
class Query:
    qid: int
    arrival: float               # seconds
    complexity_high: bool
    joint_reasoning: bool
    pieces: int
    summary_range: tuple
    query_len: int
    config: Optional[dict] = None
    admitted: Optional[float] = None
    finished: Optional[float] = None
    pending: int = 0             # unfinished calls of the current phase


@dataclasses.dataclass
class Call:
    query: Query
    prompt: int                  # prompt tokens
    decode: int                  # tokens to generate
    kind: str                    # "stuff", "mapper", "reduce", "rerank"
    blocks: List[int] = dataclasses.field(default_factory=list)
    kv_len: int = 0
    done_tokens: int = 0


def synthetic_queries(n: int, rate: float, seed: int, query_len=(32, 128)):
    """n queries with Poisson arrivals at `rate` per second and random profiles
    (complexity, joint reasoning, 1-10 pieces of information, a summary length
    range inside 30-200 tokens)."""
    r = np.random.Generator(np.random.PCG64(seed))
    t = np.cumsum(r.exponential(1.0 / rate, size=n))
    out = []
    for i in range(n):
        lo = int(r.integers(30, 120))
        out.append(Query(i, float(t[i]), bool(r.integers(2)), bool(r.integers(2)),
                         int(r.integers(1, 11)), (lo, int(min(200, lo + r.integers(0, 80)))),
                         int(r.integers(query_len[0], query_len[1] + 1))))
    return out


class Engine:
    def __init__(self, hq=32, hkv=8, d=128, layers=32, chunk_len=512, answer_len=32,
                 kv_budget_bytes=16 << 30, device="cuda", seed=0):
        self.hq, self.hkv, self.d = hq, hkv, d
        self.chunk_len, self.answer_len = chunk_len, answer_len
        self.bpt = 2 * layers * hkv * d * 2            # bf16 K and V of every layer
        self.budget = kv_budget_bytes
        self.used = 0
        self.dev = torch.device(device)
        self.scale = 1.0 / math.sqrt(d)
        self.num_blocks = kv_budget_bytes // (BLOCK * self.bpt) + 1
        shape = (self.num_blocks, hkv, BLOCK, d)
        self.k_cache = torch.zeros(shape, dtype=torch.bfloat16, device=self.dev)
        self.v_cache = torch.zeros(shape, dtype=torch.bfloat16, device=self.dev)
        self.free_blocks = list(range(self.num_blocks - 1, -1, -1))
        self.gen = torch.Generator(device=self.dev)
        self.gen.manual_seed(seed)
        self.running: List[Call] = []
        self.queued_calls: List[Call] = []
        self.ws = None
        self.stats = dict(prefill_launches=0, decode_launches=0, kv_writes=0, prefill_tokens=0,
                          decode_tokens=0, configs={}, fallbacks=0, no_fit_waits=0)

    # -- memory: a call holds whole pages for its prompt and generated tokens --
    def _call_bytes(self, c: Call) -> int:
        return (c.prompt + c.decode + BLOCK - 1) // BLOCK * BLOCK * self.bpt

    def _take_blocks(self, c: Call, upto_tokens: int):
        for _ in range((upto_tokens + BLOCK - 1) // BLOCK - len(c.blocks)):
            c.blocks.append(self.free_blocks.pop())

    def _release(self, c: Call):
        self.free_blocks.extend(c.blocks)
        c.blocks = []
        self.used -= self._call_bytes(c)

    def _rand(self, *shape):
        return torch.randn(shape, generator=self.gen, device=self.dev).to(torch.bfloat16)

    # -- admission ------------------------------------------------------------
    def _planned_calls(self, q: Query, method: str, kind: str) -> List[Call]:
        """The LLM calls of one synthesis phase, with the prompt and decode
        lengths rag_plan_prompts gives for this query and configuration."""
        cfg = q.config
        cu, dec = binding.rag_plan_prompts(method, [q.query_len], [cfg["num_chunks"]],
                                           self.chunk_len, cfg["intermediate_length"],
                                           self.answer_len)
        return [Call(q, cu[i + 1] - cu[i], dec[i], kind) for i in range(len(dec))]

    def _first_calls(self, q: Query) -> List[Call]:
        m = q.config["method"]
        if m == "stuff":
            calls = self._planned_calls(q, "stuff", "stuff")
        elif m == "map_rerank":
            calls = self._planned_calls(q, "map_rerank", "rerank")
        else:
            calls = self._planned_calls(q, "map_reduce_map", "mapper")
        q.pending = len(calls)
        return calls

    def _try(self, c: Call, new: List[Call]) -> bool:
        if self.used + self._call_bytes(c) <= self.budget:
            self.used += self._call_bytes(c)
            new.append(c)
            return True
        return False

    def admit(self, waiting: List[Query], now: float) -> List[Call]:
        """Queued calls first (remaining mappers, reduce calls), then arrived
        queries in order while the planner finds a configuration that fits."""
        new: List[Call] = []
        self.queued_calls = [c for c in self.queued_calls if not self._try(c, new)]
        while waiting and waiting[0].arrival <= now:
            q = waiting[0]
            cfg = binding.rag_choose_config(q.complexity_high, q.joint_reasoning, q.pieces,
                                            q.summary_range, q.query_len, self.chunk_len,
                                            self.answer_len, self.bpt, self.budget - self.used)
            if cfg is None:
                self.stats["no_fit_waits"] += 1
                break
            waiting.pop(0)
            q.config, q.admitted = cfg, now
            self.stats["configs"][cfg["method"]] = self.stats["configs"].get(cfg["method"], 0) + 1
            self.stats["fallbacks"] += int(cfg["fallback"])
            for c in self._first_calls(q):
                if not self._try(c, new):
                    self.queued_calls.append(c)       # mappers enter as memory frees
        return new

    # -- one iteration: operands and metadata first, then the timed launches --
    def prepare(self, new: List[Call]) -> dict:
        ops = {}
        if new:
            lens = [c.prompt for c in new]
            cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
            T = int(cu[-1])
            slots = []
            for c in new:
                self._take_blocks(c, c.prompt)
                j = np.arange(c.prompt)
                b = np.asarray(c.blocks, dtype=np.int64)
                slots.append(b[j // BLOCK] * BLOCK + j % BLOCK)
                c.kv_len = c.prompt
            ops["prefill"] = dict(
                q=self._rand(T, self.hq, self.d), k=self._rand(T, self.hkv, self.d),
                v=self._rand(T, self.hkv, self.d),
                o=torch.empty((T, self.hq, self.d), dtype=torch.bfloat16, device=self.dev),
                cu=torch.from_numpy(cu).to(self.dev), max_len=int(max(lens)),
                slots=torch.from_numpy(np.concatenate(slots).astype(np.int32)).to(self.dev))
            self.stats["prefill_tokens"] += T
            self.running.extend(new)
        if self.running:
            S = len(self.running)
            slots = []
            for c in self.running:
                self._take_blocks(c, c.kv_len + 1)
                slots.append(c.blocks[c.kv_len // BLOCK] * BLOCK + c.kv_len % BLOCK)
                c.kv_len += 1
            mb = max(len(c.blocks) for c in self.running)
            table = np.zeros((S, mb), dtype=np.int32)
            for i, c in enumerate(self.running):
                table[i, :len(c.blocks)] = c.blocks
            nbytes = binding.rag_attn_decode_workspace_size(S, self.hq, self.hkv, self.d, mb)
            if nbytes > 0 and (self.ws is None or self.ws.numel() < nbytes):
                self.ws = torch.zeros(nbytes, dtype=torch.uint8, device=self.dev)
            ops["decode"] = dict(
                kn=self._rand(S, self.hkv, self.d), vn=self._rand(S, self.hkv, self.d),
                q=self._rand(S, self.hq, self.d),
                o=torch.empty((S, self.hq, self.d), dtype=torch.bfloat16, device=self.dev),
                slots=torch.tensor(slots, dtype=torch.int32, device=self.dev),
                table=torch.from_numpy(table).to(self.dev),
                kv=torch.tensor([c.kv_len for c in self.running], dtype=torch.int32,
                                device=self.dev),
                ws=self.ws if nbytes > 0 else None)
            self.stats["decode_tokens"] += S
        return ops

    def launch(self, ops: dict):
        p = ops.get("prefill")
        if p:
            binding.rag_attn_prefill_varlen(p["q"], p["k"], p["v"], p["o"], None, p["cu"], p["cu"],
                                            p["max_len"], p["max_len"], self.scale, True)
            binding.rag_kv_cache_write(p["k"], p["v"], self.k_cache, self.v_cache, p["slots"])
            self.stats["prefill_launches"] += 1
            self.stats["kv_writes"] += 1
        d = ops.get("decode")
        if d:
            binding.rag_kv_cache_write(d["kn"], d["vn"], self.k_cache, self.v_cache, d["slots"])
            binding.rag_attn_decode_paged(d["q"], self.k_cache, self.v_cache, d["o"], d["table"],
                                          d["kv"], self.scale, workspace=d["ws"])
            self.stats["decode_launches"] += 1
            self.stats["kv_writes"] += 1

    def retire(self, now: float):
        keep = []
        for c in self.running:
            c.done_tokens += 1
            if c.done_tokens < c.decode:
                keep.append(c)
                continue
            self._release(c)
            q = c.query
            q.pending -= 1
            if q.pending > 0:
                continue
            if c.kind == "mapper":                     # all summaries written: reduce
                reduce = self._planned_calls(q, "map_reduce_reduce", "reduce")
                q.pending = len(reduce)
                self.queued_calls.extend(reduce)
            else:
                q.finished = now
        self.running = keep


def run_stream(queries: List[Query], engine: Engine, max_iters: int = 1000000) -> Dict:
    """Drive the queries through the engine; returns timing and statistics."""
    waiting = sorted(queries, key=lambda q: q.arrival)
    now = 0.0
    gpu_s = 0.0
    iters = 0
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    while (waiting or engine.running or engine.queued_calls) and iters < max_iters:
        if not engine.running and not engine.queued_calls and waiting and waiting[0].arrival > now:
            now = waiting[0].arrival                  # idle until the next arrival
        new = engine.admit(waiting, now)
        if not new and not engine.running:
            raise RuntimeError("a call can never fit in the KV budget")
        ops = engine.prepare(new)
        torch.cuda.synchronize()
        e0.record()
        engine.launch(ops)
        e1.record()
        torch.cuda.synchronize()
        dt = e0.elapsed_time(e1) / 1e3
        gpu_s += dt
        now += dt
        engine.retire(now)
        iters += 1
    done = [q for q in queries if q.finished is not None]
    lat = sorted(q.finished - q.arrival for q in done)
    return dict(queries=len(queries), completed=len(done), iterations=iters,
                gpu_seconds=round(gpu_s, 4), sim_seconds=round(now, 4),
                mean_latency_s=round(float(np.mean(lat)), 4) if lat else None,
                p90_latency_s=round(float(lat[int(0.9 * (len(lat) - 1))]), 4) if lat else None,
                **engine.stats)
