"""MI355X (gfx950) attention for the LLM synthesis step of a
configuration-adaptive RAG system (METIS, arXiv 2412.10543).

  librag_attn.so   HIP kernels + C ABI (include/rag_attn.h), built by build.py
  binding          ctypes binding with the C ABI's names (loads the library)
  workloads        seeded synthetic inputs (no attention arithmetic)

The binding is imported lazily so that the input generators can be used
without the built library.
"""
import importlib

__all__ = ["binding", "workloads", "build"]


def __getattr__(name):
    if name in ("binding", "workloads", "build"):
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
