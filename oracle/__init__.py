"""The oracle: a plain, slow, fp64 CPU implementation of what the RAG-synthesis
attention path computes.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
bench's ``cpu_baseline`` leg may import, call, link or run anything in this
directory.  The GPU library never calls it and it never calls the GPU library;
the two share no code.  Inputs reach both sides from the seeded generators in
``paper_2412_10543_amd/workloads.py``, which hold none of the method's
arithmetic.

Contents
  attn_oracle.c  fp64 attention from its definition (packed varlen prefill,
                 paged decode / chunked prefill, sampled rows), OpenMP over
                 (sequence, head)
  attention.py   ctypes wrapper, exact bf16 -> fp64 widening, gcc build step
  planner.py     prompt lengths per synthesis method (Sec. "RAG systems and
                 configurations")
  kvcache.py     paged KV-cache write (token -> page, offset by its slot)
  scheduler.py   configuration pruning (Algorithm 1) and memory-aware choice
  awq.py         group-quantized int4-weight GEMM (dequantize, multiply)

Pins: ``tests/test_oracle_pins.py`` checks the oracle against brute force on
tiny inputs, closed forms and invariants; ``tests/test_oracle_mutants.py``
plants mistakes in a copy of the C source and checks that the pins catch each
one.
"""
from .attention import Oracle, bf16_bits_to_f64, build, default  # noqa: F401
from .awq import awq_gemm, dequantize  # noqa: F401
from .kvcache import slots_from_block_table, write_kv_cache  # noqa: F401
from .planner import plan_prompts  # noqa: F401
