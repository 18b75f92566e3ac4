"""Seeded synthetic inputs for the RAG-synthesis attention path.

This module is shared by the GPU path's tests and bench and by the oracle's
tests.  It holds none of the method's arithmetic: it draws the per-query knob
values (query length, num_chunks, ...), Q/K/V values and the physical layout of
a paged KV pool.  Prompt lengths are NOT computed here; the GPU library's
planner (``rag_plan_prompts``) and the oracle's planner each derive them from
the knob values.

Value recipe: Q, K, V ~ N(0, 1) drawn in fp32 from a seeded torch generator and
rounded to bf16 (round-to-nearest-even).  The paper runs on four QA datasets
(Squad, Musique, KG RAG FinSec, QMSUM; Sec. "Evaluation", Table
"tab:table_input": inputs of 0.4K-12K tokens); they are not used, the shapes
below stand in for them.

The five workloads (sizes from the served models of Sec. "Setup": a 7B model
with 32 query heads, 8 KV heads and head size 128, and the per-GPU share of a
70B model with 64 query heads and 8 KV heads):
  tiny      stuff, 1 query: 32 query tokens + 2 chunks x 128 tokens;
            Hq=4, Hkv=2, d=64; 16 decode steps
  stuff7b   stuff, 16 queries: 64 query tokens + n ~ U{5..20} chunks x 512;
            Hq=32, Hkv=8, d=128; 128 decode steps
  mapred7b  map_reduce map phase: 16 queries x 20 chunks, each mapper prompt
            64 + 512 tokens; Hq=32, Hkv=8, d=128; intermediate_length 64
  long70b   stuff, 4 queries: 64 query tokens + 35 chunks x 1024;
            Hq=64, Hkv=8, d=128; 256 decode steps
  mixed     one batch: 256 decoding sequences with kv lengths log-uniform in
            [1024, 32768] and 4 chunked-prefill pieces of 2048 tokens whose
            prior context is U{0..8192}; Hq=32, Hkv=8, d=128
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np
import torch

BLOCK_SIZE = 16


@dataclasses.dataclass
class Workload:
    name: str
    method: str                 # synthesis method (planner spelling)
    query_lens: List[int]
    num_chunks: List[int]
    chunk_len: int
    intermediate_length: int
    answer_len: int             # decode steps of the answer calls
    hq: int
    hkv: int
    d: int
    seed: int
    block_size: int = BLOCK_SIZE

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)


@dataclasses.dataclass
class MixedWorkload:
    name: str
    decode_kv_lens: List[int]   # one query row each
    piece_prior: List[int]      # prior context of each chunked-prefill piece
    piece_len: int
    hq: int
    hkv: int
    d: int
    seed: int
    block_size: int = BLOCK_SIZE

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def tiny() -> Workload:
    return Workload("tiny", "stuff", [32], [2], 128, 0, 16, 4, 2, 64, seed=1001)


def stuff7b() -> Workload:
    r = _rng(1002)
    n = [int(x) for x in r.integers(5, 21, size=16)]      # U{5..20}
    return Workload("stuff7b", "stuff", [64] * 16, n, 512, 0, 128, 32, 8, 128,
                    seed=1002)


def mapred7b() -> Workload:
    return Workload("mapred7b", "map_reduce_map", [64] * 16, [20] * 16, 512, 64,
                    0, 32, 8, 128, seed=1003)


def long70b() -> Workload:
    return Workload("long70b", "stuff", [64] * 4, [35] * 4, 1024, 0, 256, 64, 8,
                    128, seed=1004)


def mixed() -> MixedWorkload:
    r = _rng(1005)
    kv = np.rint(np.exp(r.uniform(math.log(1024), math.log(32768), size=256)))
    prior = r.integers(0, 8193, size=4)                      # U{0..8192}
    return MixedWorkload("mixed", [int(x) for x in kv], [int(x) for x in prior],
                         2048, 32, 8, 128, seed=1005)


WORKLOADS = {"tiny": tiny, "stuff7b": stuff7b, "mapred7b": mapred7b,
             "long70b": long70b, "mixed": mixed}


# --------------------------------------------------------------------------
# value generators
# --------------------------------------------------------------------------
def normal_bf16(shape, seed: int, device="cpu", scale: float = 1.0) -> torch.Tensor:
    """N(0, scale^2) drawn in fp32 from a seeded generator, rounded to bf16."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if scale != 1.0:
        x.mul_(scale)
    return x.to(torch.bfloat16)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> numpy uint16 bit patterns (host copy)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


@dataclasses.dataclass
class PagedPool:
    k_cache: torch.Tensor        # [num_blocks, hkv, bs, d] bf16
    v_cache: torch.Tensor
    block_tables: torch.Tensor   # [S, max_blocks] int32
    kv_lens: List[int]           # tokens stored per sequence
    num_blocks: int


def paged_pool(kv_lens, hkv: int, d: int, seed: int, block_size: int = BLOCK_SIZE,
               device="cpu", pool_factor: float = 1.25, poison: bool = True,
               max_blocks: Optional[int] = None, value_scale: float = 1.0) -> PagedPool:
    """A paged KV pool holding kv_lens[s] random tokens for each sequence.

    Physical blocks are a seeded random permutation of a pool ``pool_factor``
    times larger than needed; unused blocks, the tail slots of each sequence's
    last block and the unused block-table entries are poisoned (NaN values,
    table entries pointing at a poisoned block) so that any read outside the
    visible keys shows up in the result.
    """
    bs = block_size
    nblk = [(n + bs - 1) // bs for n in kv_lens]
    need = sum(nblk)
    num_blocks = max(int(math.ceil(need * pool_factor)), need + 1)
    mb = max(nblk) if max_blocks is None else max_blocks
    r = _rng(seed)
    perm = r.permutation(num_blocks)
    spare = int(perm[need]) if need < num_blocks else 0
    table = np.full((len(kv_lens), max(mb, 1)), spare, dtype=np.int32)
    pos = 0
    for s, nb in enumerate(nblk):
        table[s, :nb] = perm[pos:pos + nb]
        pos += nb
    shape = (num_blocks, hkv, bs, d)
    k = normal_bf16(shape, seed * 7 + 1, device, value_scale)
    v = normal_bf16(shape, seed * 7 + 2, device, 1.0)
    if poison:
        used = np.zeros((num_blocks, bs), dtype=bool)
        for s, n in enumerate(kv_lens):
            for b in range(nblk[s]):
                used[table[s, b], : min(bs, n - b * bs)] = True
        mask = torch.from_numpy(~used).to(device)[:, None, :, None]
        nan = torch.tensor(float("nan"), dtype=torch.bfloat16, device=device)
        k = torch.where(mask, nan, k)
        v = torch.where(mask, nan, v)
    return PagedPool(k.contiguous(), v.contiguous(),
                     torch.from_numpy(table).to(device), list(kv_lens), num_blocks)


# --------------------------------------------------------------------------
# group-quantized int4 weights
# --------------------------------------------------------------------------
AWQ_GROUP = 128
# Linear layers of the 7B model (hidden 4096, MLP 14336, 32 q / 8 kv heads of
# 128): (name, K, N) with y[M, N] = x[M, K] W[K, N].
AWQ_LAYERS_7B = (("qkv_proj", 4096, 6144), ("o_proj", 4096, 4096),
                 ("gate_up_proj", 4096, 28672), ("down_proj", 14336, 4096))


@dataclasses.dataclass
class AwqProblem:
    x: torch.Tensor        # [M, K] bf16 on the requested device
    codes: np.ndarray      # uint8 [K, N], 0..15
    zeros: np.ndarray      # uint8 [K / 128, N], 0..15
    scales: torch.Tensor   # bf16 [K / 128, N] (host)


def awq_problem(M: int, N: int, K: int, seed: int, device="cpu") -> AwqProblem:
    """x ~ N(0, 1) in bf16; codes and zero points uniform on 0..15; scales
    uniform in [0.5, 1.5] / (6.5 sqrt(K)) rounded to bf16, so that the weights
    have a spread near 1 / sqrt(K) (the code minus zero point has standard
    deviation about 6.5) and outputs stay of order 1."""
    rng = _rng(seed)
    codes = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
    groups = K // AWQ_GROUP
    zeros = rng.integers(0, 16, size=(groups, N), dtype=np.uint8)
    s = rng.uniform(0.5, 1.5, size=(groups, N)) / (6.5 * np.sqrt(K))
    scales = torch.from_numpy(s.astype(np.float32)).to(torch.bfloat16)
    x = normal_bf16((M, K), seed + 1, device)
    return AwqProblem(x, codes, zeros, scales)
