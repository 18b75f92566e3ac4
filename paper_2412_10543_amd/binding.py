"""Thin Python binding of librag_attn.so (the C ABI in include/rag_attn.h).

Argument marshalling only: every step of the attention path runs in the HIP
library.  Tensors are torch tensors on the GPU (torch supplies device memory
and the current HIP stream); shapes, dtypes and contiguity are checked here
and everything else is left to the library's own validation.  There is no
fallback: if the library is missing or was built for another target, loading
raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

LIBRARY = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librag_attn.so")

RAG_NO_FIT = 1
RAG_OK = 0
RAG_ERR_INVALID_ARG = -1
RAG_ERR_UNSUPPORTED = -2
RAG_ERR_WORKSPACE = -3
RAG_ERR_HIP = -4

RAG_STUFF = 0
RAG_MAP_REDUCE_MAP = 1
RAG_MAP_REDUCE_REDUCE = 2
RAG_MAP_RERANK = 3
METHOD_CODES = {"stuff": RAG_STUFF, "map_reduce_map": RAG_MAP_REDUCE_MAP,
                "map_reduce_reduce": RAG_MAP_REDUCE_REDUCE, "map_rerank": RAG_MAP_RERANK}


class RagError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"rag_attn status {status}: {message}")
        self.status = status


_i32 = ctypes.c_int32
_i32p = ctypes.POINTER(ctypes.c_int32)
_vp = ctypes.c_void_p
_lib = None


def exported_symbols():
    return ["rag_abi_version", "rag_last_error", "rag_attn_prefill_varlen",
            "rag_attn_prefill_varlen_kvcache", "rag_attn_decode_paged_append",
            "rag_attn_decode_num_splits", "rag_attn_decode_workspace_size",
            "rag_attn_decode_paged", "rag_attn_decode_paged_noalloc", "rag_kv_cache_write", "rag_plan_prompts",
            "rag_prune_config_space", "rag_config_kv_bytes", "rag_choose_config",
            "rag_device_free_memory", "rag_awq_pack_weights", "rag_awq_workspace_size",
            "rag_awq_gemm"]


class QueryProfile(ctypes.Structure):
    _fields_ = [("complexity_high", ctypes.c_int32), ("joint_reasoning", ctypes.c_int32),
                ("pieces", ctypes.c_int32), ("summary_len_min", ctypes.c_int32),
                ("summary_len_max", ctypes.c_int32)]


class ConfigSpace(ctypes.Structure):
    _fields_ = [("methods", ctypes.c_uint32), ("num_chunks_min", ctypes.c_int32),
                ("num_chunks_max", ctypes.c_int32), ("intermediate_length_min", ctypes.c_int32),
                ("intermediate_length_max", ctypes.c_int32)]


class RequestShape(ctypes.Structure):
    _fields_ = [("query_len", ctypes.c_int32), ("chunk_len", ctypes.c_int32),
                ("answer_len", ctypes.c_int32), ("kv_bytes_per_token", ctypes.c_int64)]


class Config(ctypes.Structure):
    _fields_ = [("method", ctypes.c_int32), ("num_chunks", ctypes.c_int32),
                ("intermediate_length", ctypes.c_int32), ("fallback", ctypes.c_int32),
                ("kv_bytes", ctypes.c_int64)]


def lib():
    """Load (once) and return the ctypes handle of librag_attn.so."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIBRARY):
        raise ImportError(f"{LIBRARY} is not built; run __graft_entry__.build() or "
                          "python -m paper_2412_10543_amd.build")
    L = ctypes.CDLL(LIBRARY)
    L.rag_abi_version.restype = ctypes.c_int
    L.rag_last_error.restype = ctypes.c_char_p
    L.rag_attn_prefill_varlen.restype = ctypes.c_int
    L.rag_attn_prefill_varlen.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32,
                                          _i32, _i32, _i32, ctypes.c_float, _i32, _vp]
    L.rag_attn_prefill_varlen_kvcache.restype = ctypes.c_int
    L.rag_attn_prefill_varlen_kvcache.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32,
                                                  _i32, _i32, ctypes.c_float, _vp, _vp, _vp,
                                                  _i32, _i32, _vp]
    L.rag_attn_decode_paged_append.restype = ctypes.c_int
    L.rag_attn_decode_paged_append.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32,
                                               _i32, _i32, _i32, _i32, _i32, ctypes.c_float,
                                               _i32, _vp, ctypes.c_size_t, _vp]
    L.rag_attn_decode_num_splits.restype = _i32
    L.rag_attn_decode_num_splits.argtypes = [_i32, _i32, _i32, _i32, _i32]
    L.rag_attn_decode_workspace_size.restype = ctypes.c_size_t
    L.rag_attn_decode_workspace_size.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32, _i32]
    L.rag_attn_decode_paged.restype = ctypes.c_int
    L.rag_attn_decode_paged.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32,
                                        _i32, _i32, _i32, _i32, _i32, _i32, ctypes.c_float,
                                        _i32, _vp, ctypes.c_size_t, _vp]
    L.rag_attn_decode_paged_noalloc.restype = ctypes.c_int
    L.rag_attn_decode_paged_noalloc.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32,
                                                _i32, _i32, _i32, _i32, _i32, _i32, _i32,
                                                ctypes.c_float, _i32, _vp]
    L.rag_kv_cache_write.restype = ctypes.c_int
    L.rag_kv_cache_write.argtypes = [_vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp]
    L.rag_prune_config_space.restype = ctypes.c_int
    L.rag_prune_config_space.argtypes = [ctypes.POINTER(QueryProfile), ctypes.POINTER(ConfigSpace)]
    L.rag_config_kv_bytes.restype = ctypes.c_int64
    L.rag_config_kv_bytes.argtypes = [_i32, _i32, _i32, ctypes.POINTER(RequestShape)]
    L.rag_choose_config.restype = ctypes.c_int
    L.rag_choose_config.argtypes = [ctypes.POINTER(QueryProfile), ctypes.POINTER(RequestShape),
                                    ctypes.c_int64, ctypes.POINTER(Config)]
    L.rag_device_free_memory.restype = ctypes.c_int
    L.rag_device_free_memory.argtypes = [ctypes.POINTER(ctypes.c_size_t),
                                         ctypes.POINTER(ctypes.c_size_t)]
    L.rag_awq_pack_weights.restype = ctypes.c_int
    L.rag_awq_pack_weights.argtypes = [_vp, _i32, _i32, _i32, _vp]
    L.rag_awq_workspace_size.restype = ctypes.c_size_t
    L.rag_awq_workspace_size.argtypes = [_i32, _i32, _i32, _i32]
    L.rag_awq_gemm.restype = ctypes.c_int
    L.rag_awq_gemm.argtypes = [_vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _vp,
                               ctypes.c_size_t, _vp]
    L.rag_plan_prompts.restype = ctypes.c_int
    L.rag_plan_prompts.argtypes = [ctypes.c_int, _i32, _i32p, _i32p, _i32, _i32, _i32, _i32p,
                                   _i32, _i32p, _i32p]
    _lib = L
    return L


def _check(status: int):
    if status != RAG_OK:
        raise RagError(status, lib().rag_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _need(t, dtype, name, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions")


def rag_abi_version() -> int:
    return lib().rag_abi_version()


def rag_last_error() -> str:
    return lib().rag_last_error().decode()


def rag_attn_prefill_varlen(q, k, v, o, lse, cu_seqlens_q, cu_seqlens_k, max_seqlen_q,
                            max_seqlen_k, softmax_scale, causal=True, stream=None) -> None:
    """q, o [Tq, Hq, d]; k, v [Tk, Hkv, d] bf16; lse fp32 [Hq, Tq] or None;
    cu_seqlens_* int32 [S+1] on the GPU."""
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (o, "o")):
        _need(t, torch.bfloat16, n, 3)
    _need(cu_seqlens_q, torch.int32, "cu_seqlens_q", 1)
    _need(cu_seqlens_k, torch.int32, "cu_seqlens_k", 1)
    if lse is not None:
        _need(lse, torch.float32, "lse", 2)
    _check(lib().rag_attn_prefill_varlen(
        _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(cu_seqlens_q), _ptr(cu_seqlens_k),
        cu_seqlens_q.numel() - 1, int(max_seqlen_q), int(max_seqlen_k), q.shape[1], k.shape[1],
        q.shape[2], float(softmax_scale), int(bool(causal)), _stream(stream)))


def rag_attn_prefill_varlen_kvcache(q, k, v, o, lse, cu_seqlens, max_seqlen, softmax_scale,
                                    k_cache, v_cache, slot_mapping, stream=None) -> None:
    """Causal prompt prefill that also writes K/V into the paged cache.
    q, o [T, Hq, d]; k, v [T, Hkv, d] bf16; cu_seqlens int32 [S+1]; caches
    [num_blocks, Hkv, 16, d] bf16; slot_mapping int32 [T] (negative = skip)."""
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (o, "o")):
        _need(t, torch.bfloat16, n, 3)
    for t, n in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        _need(t, torch.bfloat16, n, 4)
    _need(cu_seqlens, torch.int32, "cu_seqlens", 1)
    _need(slot_mapping, torch.int32, "slot_mapping", 1)
    if lse is not None:
        _need(lse, torch.float32, "lse", 2)
    _check(lib().rag_attn_prefill_varlen_kvcache(
        _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(cu_seqlens), cu_seqlens.shape[0] - 1,
        int(max_seqlen), q.shape[1], k.shape[1], q.shape[2], float(softmax_scale),
        _ptr(k_cache), _ptr(v_cache), _ptr(slot_mapping), k_cache.shape[0], k_cache.shape[2],
        _stream(stream)))


def rag_attn_decode_paged_append(q, k_new, v_new, k_cache, v_cache, o, block_tables, kv_lens,
                                 softmax_scale, num_splits=0, workspace=None, stream=None):
    """One decode step that appends each row's new token (k_new, v_new
    [S, Hkv, d]) to the cache at key kv_lens[s] - 1 and attends it."""
    for t, n in ((q, "q"), (o, "o"), (k_new, "k_new"), (v_new, "v_new")):
        _need(t, torch.bfloat16, n, 3)
    for t, n in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        _need(t, torch.bfloat16, n, 4)
    _need(block_tables, torch.int32, "block_tables", 2)
    _need(kv_lens, torch.int32, "kv_lens", 1)
    ws_bytes = 0
    if workspace is not None:
        if not workspace.is_cuda or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous GPU tensor")
        ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().rag_attn_decode_paged_append(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(o),
        _ptr(block_tables), _ptr(kv_lens), block_tables.shape[0], block_tables.shape[1],
        k_cache.shape[0], q.shape[1], k_cache.shape[1], q.shape[2], k_cache.shape[2],
        float(softmax_scale), int(num_splits), _ptr(workspace), ws_bytes, _stream(stream)))


def rag_attn_decode_num_splits(num_decode_seqs, num_kv_heads, max_blocks_per_seq,
                               block_size=16, num_splits=0) -> int:
    return lib().rag_attn_decode_num_splits(num_decode_seqs, num_kv_heads, max_blocks_per_seq,
                                            block_size, num_splits)


def rag_attn_decode_workspace_size(num_decode_seqs, num_q_heads, num_kv_heads, head_dim,
                                   max_blocks_per_seq, block_size=16, num_splits=0) -> int:
    return lib().rag_attn_decode_workspace_size(num_decode_seqs, num_q_heads, num_kv_heads,
                                                head_dim, max_blocks_per_seq, block_size,
                                                num_splits)


def rag_attn_decode_paged(q, k_cache, v_cache, o, block_tables, kv_lens, softmax_scale,
                          cu_seqlens_q=None, num_decode_seqs=None, max_seqlen_q=1,
                          num_splits=0, workspace=None, stream=None) -> None:
    """q, o [Tq, Hq, d]; caches [num_blocks, Hkv, 16, d] bf16; block_tables
    int32 [S, max_blocks]; kv_lens int32 [S]; cu_seqlens_q int32 [S+1] or
    None; workspace a zero-initialised GPU tensor (torch.zeros, uint8) of
    rag_attn_decode_workspace_size bytes, or None when that size is 0."""
    for t, n in ((q, "q"), (o, "o")):
        _need(t, torch.bfloat16, n, 3)
    for t, n in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        _need(t, torch.bfloat16, n, 4)
    _need(block_tables, torch.int32, "block_tables", 2)
    _need(kv_lens, torch.int32, "kv_lens", 1)
    if cu_seqlens_q is not None:
        _need(cu_seqlens_q, torch.int32, "cu_seqlens_q", 1)
    num_seqs = block_tables.shape[0]
    if num_decode_seqs is None:
        num_decode_seqs = num_seqs
    ws_bytes = 0
    if workspace is not None:
        if not workspace.is_cuda or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous GPU tensor")
        ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().rag_attn_decode_paged(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(o), _ptr(block_tables), _ptr(kv_lens),
        _ptr(cu_seqlens_q), num_seqs, int(num_decode_seqs), block_tables.shape[1],
        int(max_seqlen_q), k_cache.shape[0], q.shape[1], k_cache.shape[1], q.shape[2],
        k_cache.shape[2], float(softmax_scale), int(num_splits), _ptr(workspace), ws_bytes,
        _stream(stream)))


def rag_attn_decode_paged_noalloc(q, k_cache, v_cache, o, block_tables, kv_lens, softmax_scale,
                                  cu_seqlens_q=None, num_decode_seqs=None, max_seqlen_q=1,
                                  num_splits=0, stream=None) -> None:
    """rag_attn_decode_paged with the library's static scratch instead of a
    workspace (allocates nothing)."""
    for t, n in ((q, "q"), (o, "o")):
        _need(t, torch.bfloat16, n, 3)
    for t, n in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        _need(t, torch.bfloat16, n, 4)
    _need(block_tables, torch.int32, "block_tables", 2)
    _need(kv_lens, torch.int32, "kv_lens", 1)
    if cu_seqlens_q is not None:
        _need(cu_seqlens_q, torch.int32, "cu_seqlens_q", 1)
    num_seqs = block_tables.shape[0]
    if num_decode_seqs is None:
        num_decode_seqs = num_seqs
    _check(lib().rag_attn_decode_paged_noalloc(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(o), _ptr(block_tables), _ptr(kv_lens),
        _ptr(cu_seqlens_q), num_seqs, int(num_decode_seqs), block_tables.shape[1],
        int(max_seqlen_q), k_cache.shape[0], q.shape[1], k_cache.shape[1], q.shape[2],
        k_cache.shape[2], float(softmax_scale), int(num_splits), _stream(stream)))


def rag_kv_cache_write(k, v, k_cache, v_cache, slot_mapping, stream=None) -> None:
    """k, v [T, Hkv, d] bf16; caches [num_blocks, Hkv, 16, d] bf16; slot_mapping
    int32 [T] on the GPU (negative = skip)."""
    for t, n in ((k, "k"), (v, "v")):
        _need(t, torch.bfloat16, n, 3)
    for t, n in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        _need(t, torch.bfloat16, n, 4)
    _need(slot_mapping, torch.int32, "slot_mapping", 1)
    _check(lib().rag_kv_cache_write(
        _ptr(k), _ptr(v), _ptr(k_cache), _ptr(v_cache), _ptr(slot_mapping), k.shape[0],
        k.shape[1], k.shape[2], k_cache.shape[2], k_cache.shape[0], _stream(stream)))


def rag_plan_prompts(method, query_len, num_chunks, chunk_len, intermediate_length=0,
                     answer_len=0):
    """Host planner.  Returns (cu_seqlens list, decode_len list)."""
    code = METHOD_CODES[method] if isinstance(method, str) else int(method)
    n = len(query_len)
    ql = (_i32 * max(n, 1))(*query_len)
    nc = (_i32 * max(n, 1))(*num_chunks)
    count = _i32(0)
    L = lib()
    st = L.rag_plan_prompts(code, n, ql, nc, chunk_len, intermediate_length, answer_len, None, 0,
                            ctypes.byref(count), None)
    if st not in (RAG_OK, RAG_ERR_WORKSPACE):
        _check(st)
    cap = count.value + 1
    cu = (_i32 * cap)()
    dec = (_i32 * max(count.value, 1))()
    _check(L.rag_plan_prompts(code, n, ql, nc, chunk_len, intermediate_length, answer_len, cu,
                              cap, ctypes.byref(count), dec))
    return list(cu), list(dec)[:count.value]


# ---------------------------------------------------------------------------
# configuration planner (host only)
# ---------------------------------------------------------------------------
CONFIG_METHOD_NAMES = {RAG_STUFF: "stuff", RAG_MAP_REDUCE_MAP: "map_reduce",
                       RAG_MAP_RERANK: "map_rerank"}


def _profile(complexity_high, joint_reasoning, pieces, summary_range):
    return QueryProfile(int(bool(complexity_high)), int(bool(joint_reasoning)), int(pieces),
                        int(summary_range[0]), int(summary_range[1]))


def rag_prune_config_space(complexity_high, joint_reasoning, pieces, summary_range):
    """Algorithm 1.  Returns (method names, (chunks_min, chunks_max),
    (il_min, il_max))."""
    sp = ConfigSpace()
    _check(lib().rag_prune_config_space(
        ctypes.byref(_profile(complexity_high, joint_reasoning, pieces, summary_range)),
        ctypes.byref(sp)))
    methods = tuple(n for m, n in CONFIG_METHOD_NAMES.items() if sp.methods & (1 << m))
    return methods, (sp.num_chunks_min, sp.num_chunks_max), \
        (sp.intermediate_length_min, sp.intermediate_length_max)


def _shape(query_len, chunk_len, answer_len, bytes_per_token):
    return RequestShape(int(query_len), int(chunk_len), int(answer_len), int(bytes_per_token))


def rag_config_kv_bytes(method, num_chunks, intermediate_length, query_len, chunk_len,
                        answer_len, bytes_per_token) -> int:
    code = {v: k for k, v in CONFIG_METHOD_NAMES.items()}[method] if isinstance(method, str) \
        else int(method)
    return lib().rag_config_kv_bytes(code, int(num_chunks), int(intermediate_length),
                                     ctypes.byref(_shape(query_len, chunk_len, answer_len,
                                                         bytes_per_token)))


def rag_choose_config(complexity_high, joint_reasoning, pieces, summary_range, query_len,
                      chunk_len, answer_len, bytes_per_token, available_bytes):
    """Best-fit choice.  Returns a dict (method name, num_chunks,
    intermediate_length, kv_bytes, fallback) or None when nothing fits."""
    out = Config()
    st = lib().rag_choose_config(
        ctypes.byref(_profile(complexity_high, joint_reasoning, pieces, summary_range)),
        ctypes.byref(_shape(query_len, chunk_len, answer_len, bytes_per_token)),
        int(available_bytes), ctypes.byref(out))
    if st == RAG_NO_FIT:
        return None
    _check(st)
    return dict(method=CONFIG_METHOD_NAMES[out.method], num_chunks=out.num_chunks,
                intermediate_length=out.intermediate_length, kv_bytes=out.kv_bytes,
                fallback=bool(out.fallback))


def rag_device_free_memory():
    """(free bytes, total bytes) of the current HIP device."""
    f, t = ctypes.c_size_t(0), ctypes.c_size_t(0)
    _check(lib().rag_device_free_memory(ctypes.byref(f), ctypes.byref(t)))
    return f.value, t.value


def rag_awq_pack_weights(q, group_size: int = 128):
    """Host packer: q a numpy uint8 array [K, N] of 4-bit codes -> numpy int32
    [K // group_size, N, 16] in the kernel's order."""
    import numpy as np
    q = np.ascontiguousarray(q, dtype=np.uint8)
    if q.ndim != 2:
        raise ValueError("q must be [K, N]")
    K, N = q.shape
    out = np.empty((max(K // 128, 0), N, 16), dtype=np.int32)
    _check(lib().rag_awq_pack_weights(q.ctypes.data, K, N, int(group_size), out.ctypes.data))
    return out


def rag_awq_workspace_size(M: int, N: int, K: int, group_size: int = 128) -> int:
    return int(lib().rag_awq_workspace_size(int(M), int(N), int(K), int(group_size)))


def rag_awq_gemm(x, qweight, scales, zeros, y, workspace, group_size: int = 128,
                 stream=None) -> None:
    """x [M, K] bf16; qweight int32 [K/128, N, 16] (rag_awq_pack_weights);
    scales bf16 [K/128, N]; zeros uint8 [K/128, N]; y [M, N] bf16 output;
    workspace a GPU uint8 tensor of rag_awq_workspace_size bytes, zero-filled
    once before its first use (every call leaves its counters zero again)."""
    _need(x, torch.bfloat16, "x", 2)
    _need(qweight, torch.int32, "qweight", 3)
    _need(scales, torch.bfloat16, "scales", 2)
    _need(zeros, torch.uint8, "zeros", 2)
    _need(y, torch.bfloat16, "y", 2)
    M, K = x.shape
    N = y.shape[1]
    if y.shape[0] != M or qweight.shape != (K // 128, N, 16) or \
            scales.shape != (K // 128, N) or zeros.shape != (K // 128, N):
        raise ValueError("awq gemm: inconsistent shapes")
    ws_bytes = 0
    if workspace is not None:
        if not workspace.is_cuda or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous GPU tensor")
        ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().rag_awq_gemm(_ptr(x), _ptr(qweight), _ptr(scales), _ptr(zeros), _ptr(y), M, N,
                              K, int(group_size), _ptr(workspace), ws_bytes, _stream(stream)))
