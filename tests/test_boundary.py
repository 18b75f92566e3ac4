"""The C ABI on the CPU: the library loads, exports every function the header
declares, rejects bad host arguments with the documented status before
enqueueing anything, and its prompt planner matches the oracle's.

No call here reaches a kernel launch: every call either fails validation or is
a documented no-op (num_seqs == 0), so no GPU is needed.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import plan_prompts as oracle_plan
from paper_2412_10543_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rag_attn.h")

pytestmark = pytest.mark.skipif(not os.path.exists(binding.LIBRARY),
                                reason="librag_attn.so not built")

FAKE = 0x100000  # 16- and 256-byte aligned address; never dereferenced on these paths


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rag_[a-z0-9_]+)\s*\(", text)))


def test_header_declarations_exported():
    L = binding.lib()
    names = _declared()
    assert names == sorted(binding.exported_symbols())
    for n in names:
        assert hasattr(L, n), f"{n} not exported"


def test_ceiling_probe_library_exports_its_header():
    """The measurement probes (bench.py --ceilings) live in their own library;
    its header's declarations are exactly its exports, and bad arguments are
    rejected without a launch."""
    import ctypes
    from paper_2412_10543_amd import build as pb
    if not os.path.exists(pb.PROBES):
        pytest.skip("libceiling_probes.so not built")
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "ceiling_probes.h")).read(),
                  flags=re.S)
    names = sorted(set(re.findall(r"\b(rag_[a-z0-9_]+)\s*\(", text)))
    assert names == ["rag_probe_attn_pair", "rag_probe_attn_slot", "rag_probe_kv_page_read",
                     "rag_probe_mfma_loop",
                     "rag_probe_page_read", "rag_probe_softmax_mfma", "rag_probe_stream_read"]
    L = ctypes.CDLL(pb.PROBES)
    for n in names:
        assert hasattr(L, n)
    L.rag_probe_mfma_loop.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p]
    for n in ("rag_probe_mfma_loop", "rag_probe_attn_slot", "rag_probe_softmax_mfma",
              "rag_probe_attn_pair"):
        f = getattr(L, n)
        f.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
        assert f(10, 0, FAKE, None) == -1
        assert f(10, 4, None, None) == -1
        assert f(-1, 4, FAKE, None) == -1


def test_abi_version():
    assert binding.rag_abi_version() == 1


def _prefill(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=None, cu_q=FAKE, cu_k=FAKE, num_seqs=1,
             max_q=16, max_k=16, hq=4, hkv=2, d=64, scale=0.125, causal=1)
    a.update(kw)
    return binding.lib().rag_attn_prefill_varlen(
        a["q"], a["k"], a["v"], a["o"], a["lse"], a["cu_q"], a["cu_k"], a["num_seqs"],
        a["max_q"], a["max_k"], a["hq"], a["hkv"], a["d"], a["scale"], a["causal"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), binding.RAG_ERR_INVALID_ARG),
    (dict(cu_k=None), binding.RAG_ERR_INVALID_ARG),
    (dict(num_seqs=-1), binding.RAG_ERR_INVALID_ARG),
    (dict(hq=6, hkv=4), binding.RAG_ERR_INVALID_ARG),
    (dict(hkv=0), binding.RAG_ERR_INVALID_ARG),
    (dict(causal=2), binding.RAG_ERR_INVALID_ARG),
    (dict(scale=0.0), binding.RAG_ERR_INVALID_ARG),
    (dict(scale=float("nan")), binding.RAG_ERR_INVALID_ARG),
    (dict(q=FAKE + 8), binding.RAG_ERR_INVALID_ARG),
    (dict(d=96), binding.RAG_ERR_UNSUPPORTED),
    (dict(d=256), binding.RAG_ERR_UNSUPPORTED),
    (dict(num_seqs=0), binding.RAG_OK),
    (dict(max_q=0), binding.RAG_OK),
])
def test_prefill_validation(kw, status):
    assert _prefill(**kw) == status
    if status != binding.RAG_OK:
        assert binding.rag_last_error() != ""
    else:
        assert binding.rag_last_error() == ""


def _decode(**kw):
    a = dict(q=FAKE, kc=FAKE, vc=FAKE, o=FAKE, bt=FAKE, kl=FAKE, cu=None, num_seqs=4,
             num_decode=4, max_blocks=64, max_q=1, num_blocks=300, hq=32, hkv=8, d=128, bs=16,
             scale=0.088, splits=0, ws=None, ws_bytes=0)
    a.update(kw)
    return binding.lib().rag_attn_decode_paged(
        a["q"], a["kc"], a["vc"], a["o"], a["bt"], a["kl"], a["cu"], a["num_seqs"],
        a["num_decode"], a["max_blocks"], a["max_q"], a["num_blocks"], a["hq"], a["hkv"],
        a["d"], a["bs"], a["scale"], a["splits"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(kc=None), binding.RAG_ERR_INVALID_ARG),
    (dict(kl=None), binding.RAG_ERR_INVALID_ARG),
    (dict(num_seqs=-2), binding.RAG_ERR_INVALID_ARG),
    (dict(splits=-1), binding.RAG_ERR_INVALID_ARG),
    (dict(hq=12, hkv=8), binding.RAG_ERR_INVALID_ARG),
    (dict(o=FAKE + 2), binding.RAG_ERR_INVALID_ARG),
    (dict(d=80), binding.RAG_ERR_UNSUPPORTED),
    (dict(bs=32), binding.RAG_ERR_UNSUPPORTED),
    (dict(hq=64, hkv=2), binding.RAG_ERR_UNSUPPORTED),       # group of 32 > 16
    (dict(cu=FAKE, num_decode=5), binding.RAG_ERR_INVALID_ARG),
    (dict(max_blocks=0), binding.RAG_ERR_INVALID_ARG),
    (dict(splits=4), binding.RAG_ERR_WORKSPACE),               # no workspace given
    (dict(splits=4, ws=FAKE, ws_bytes=1024), binding.RAG_ERR_WORKSPACE),
    (dict(splits=4, ws=FAKE + 64, ws_bytes=1 << 30), binding.RAG_ERR_INVALID_ARG),
    (dict(num_seqs=0), binding.RAG_OK),
])
def test_decode_validation(kw, status):
    assert _decode(**kw) == status


def _decode_noalloc(**kw):
    a = dict(q=FAKE, kc=FAKE, vc=FAKE, o=FAKE, bt=FAKE, kl=FAKE, cu=None, num_seqs=4,
             num_decode=4, max_blocks=64, max_q=1, num_blocks=300, hq=32, hkv=8, d=128, bs=16,
             scale=0.088, splits=0)
    a.update(kw)
    return binding.lib().rag_attn_decode_paged_noalloc(
        a["q"], a["kc"], a["vc"], a["o"], a["bt"], a["kl"], a["cu"], a["num_seqs"],
        a["num_decode"], a["max_blocks"], a["max_q"], a["num_blocks"], a["hq"], a["hkv"],
        a["d"], a["bs"], a["scale"], a["splits"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(kc=None), binding.RAG_ERR_INVALID_ARG),
    (dict(num_seqs=-2), binding.RAG_ERR_INVALID_ARG),
    (dict(hq=12, hkv=8), binding.RAG_ERR_INVALID_ARG),
    (dict(d=80), binding.RAG_ERR_UNSUPPORTED),
    (dict(num_seqs=0), binding.RAG_OK),
    # beyond the static scratch: 4096 rows x 32 heads x 64 splits x 129 x 4 B of partials
    (dict(num_seqs=4096, num_decode=4096, splits=64), binding.RAG_ERR_WORKSPACE),
    # 16384 rows x 8 kv heads = 131072 arrival counters (> 65536)
    (dict(num_seqs=16384, num_decode=16384, max_blocks=4, splits=2), binding.RAG_ERR_WORKSPACE),
])
def test_decode_noalloc_validation(kw, status):
    """Rejected before any HIP call: the size checks come before the scratch
    set-up, so none of these needs a GPU."""
    assert _decode_noalloc(**kw) == status
    if status == binding.RAG_ERR_WORKSPACE:
        assert "no-alloc" in binding.rag_last_error()


def _prefill_kvcache(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=None, cu=FAKE, num_seqs=1, max_len=16, hq=4,
             hkv=2, d=64, scale=0.125, kc=FAKE, vc=FAKE, slots=FAKE, num_blocks=10, bs=16)
    a.update(kw)
    return binding.lib().rag_attn_prefill_varlen_kvcache(
        a["q"], a["k"], a["v"], a["o"], a["lse"], a["cu"], a["num_seqs"], a["max_len"], a["hq"],
        a["hkv"], a["d"], a["scale"], a["kc"], a["vc"], a["slots"], a["num_blocks"], a["bs"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), binding.RAG_ERR_INVALID_ARG),
    (dict(kc=None), binding.RAG_ERR_INVALID_ARG),
    (dict(slots=None), binding.RAG_ERR_INVALID_ARG),
    (dict(vc=FAKE + 8), binding.RAG_ERR_INVALID_ARG),
    (dict(num_blocks=-1), binding.RAG_ERR_INVALID_ARG),
    (dict(hq=6, hkv=4), binding.RAG_ERR_INVALID_ARG),
    (dict(bs=32), binding.RAG_ERR_UNSUPPORTED),
    (dict(d=96), binding.RAG_ERR_UNSUPPORTED),
    (dict(num_seqs=0), binding.RAG_OK),
])
def test_prefill_kvcache_validation(kw, status):
    assert _prefill_kvcache(**kw) == status


def _decode_append(**kw):
    a = dict(q=FAKE, kn=FAKE, vn=FAKE, kc=FAKE, vc=FAKE, o=FAKE, bt=FAKE, kl=FAKE, num_seqs=4,
             max_blocks=64, num_blocks=300, hq=32, hkv=8, d=128, bs=16, scale=0.088, splits=0,
             ws=None, ws_bytes=0)
    a.update(kw)
    return binding.lib().rag_attn_decode_paged_append(
        a["q"], a["kn"], a["vn"], a["kc"], a["vc"], a["o"], a["bt"], a["kl"], a["num_seqs"],
        a["max_blocks"], a["num_blocks"], a["hq"], a["hkv"], a["d"], a["bs"], a["scale"],
        a["splits"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(kn=None), binding.RAG_ERR_INVALID_ARG),
    (dict(vn=FAKE + 4), binding.RAG_ERR_INVALID_ARG),
    (dict(kc=None), binding.RAG_ERR_INVALID_ARG),
    (dict(hq=12, hkv=8), binding.RAG_ERR_INVALID_ARG),
    (dict(bs=32), binding.RAG_ERR_UNSUPPORTED),
    (dict(splits=4), binding.RAG_ERR_WORKSPACE),
    (dict(num_seqs=0), binding.RAG_OK),
])
def test_decode_append_validation(kw, status):
    assert _decode_append(**kw) == status


def _kv_write(**kw):
    a = dict(k=FAKE, v=FAKE, kc=FAKE, vc=FAKE, slots=FAKE, T=16, hkv=8, d=128, bs=16,
             num_blocks=100)
    a.update(kw)
    return binding.lib().rag_kv_cache_write(a["k"], a["v"], a["kc"], a["vc"], a["slots"], a["T"],
                                            a["hkv"], a["d"], a["bs"], a["num_blocks"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(k=None), binding.RAG_ERR_INVALID_ARG),
    (dict(slots=None), binding.RAG_ERR_INVALID_ARG),
    (dict(vc=FAKE + 8), binding.RAG_ERR_INVALID_ARG),
    (dict(T=-1), binding.RAG_ERR_INVALID_ARG),
    (dict(num_blocks=-1), binding.RAG_ERR_INVALID_ARG),
    (dict(hkv=0), binding.RAG_ERR_INVALID_ARG),
    (dict(d=96), binding.RAG_ERR_UNSUPPORTED),
    (dict(bs=8), binding.RAG_ERR_UNSUPPORTED),
    (dict(T=0, k=None, slots=None), binding.RAG_OK),          # nothing to write
])
def test_kv_write_validation(kw, status):
    assert _kv_write(**kw) == status
    if status != binding.RAG_OK:
        assert binding.rag_last_error().startswith("kv write")


def test_split_policy():
    ns = binding.rag_attn_decode_num_splits
    # one split never needs a workspace
    assert ns(2560, 8, 40, 16, 1) == 1
    assert binding.rag_attn_decode_workspace_size(2560, 32, 8, 128, 40, 16, 1) == 0
    for nd, hkv, mb in [(16, 8, 653), (4, 8, 2260), (320, 8, 40), (256, 8, 2048), (1, 2, 19),
                        (1, 1, 1), (3, 4, 7), (30, 8, 600)]:
        n = ns(nd, hkv, mb)
        assert 1 <= n <= 64
        if nd * hkv < 256:
            # balanced units: at most one per 16 pages of all rows
            assert n <= max(1, nd * mb // 16) or n <= mb
        else:
            assert n <= mb
            pps = -(-mb // n)
            assert -(-mb // pps) == n, "every split of the longest sequence is non-empty"
        ws = binding.rag_attn_decode_workspace_size(nd, hkv * 4, hkv, 128, mb)
        if n == 1:
            assert ws == 0
        else:
            assert ws >= nd * hkv * 4 * n * 129 * 4
    # uniform splits when a count is requested: every split of the longest row non-empty
    for nd, hkv, mb, req in [(16, 8, 653, 3), (1, 2, 19, 5), (2, 1, 40, 64)]:
        n = ns(nd, hkv, mb, 16, req)
        pps = -(-mb // n)
        assert n <= mb and -(-mb // pps) == n
    # requested counts are honoured up to one split per block
    assert ns(16, 8, 653, 16, 7) == 7
    assert ns(16, 8, 5, 16, 64) == 5


@pytest.mark.parametrize("method", ["stuff", "map_reduce_map", "map_reduce_reduce", "map_rerank"])
def test_planner_matches_oracle(method):
    r = np.random.Generator(np.random.PCG64(7))
    for trial in range(20):
        nq = int(r.integers(0, 12))
        ql = [int(x) for x in r.integers(1, 200, size=nq)]
        nc = [int(x) for x in r.integers(0, 36, size=nq)]
        C, IL, A = int(r.integers(1, 2048)), int(r.integers(0, 300)), int(r.integers(0, 256))
        cu, dec = binding.rag_plan_prompts(method, ql, nc, C, IL, A)
        ocu, odec, _ = oracle_plan(method, ql, nc, C, IL, A)
        assert cu == ocu and dec == odec


def test_planner_errors():
    L = binding.lib()
    n = ctypes.c_int32(0)
    one = (ctypes.c_int32 * 1)(5)
    assert L.rag_plan_prompts(9, 1, one, one, 512, 0, 0, None, 0, ctypes.byref(n), None) == \
        binding.RAG_ERR_INVALID_ARG
    neg = (ctypes.c_int32 * 1)(-1)
    assert L.rag_plan_prompts(0, 1, one, neg, 512, 0, 0, None, 0, ctypes.byref(n), None) == \
        binding.RAG_ERR_INVALID_ARG
    cu = (ctypes.c_int32 * 2)()
    assert L.rag_plan_prompts(1, 1, one, one, 512, 0, 0, cu, 2, ctypes.byref(n), None) == \
        binding.RAG_ERR_WORKSPACE  # 5 mapper calls need 6 entries
    assert n.value == 5
    big = (ctypes.c_int32 * 1)(2_000_000_000)
    many = (ctypes.c_int32 * 1)(10)
    cu2 = (ctypes.c_int32 * 2)()
    assert L.rag_plan_prompts(0, 1, big, many, 1_000_000_000, 0, 0, cu2, 2, ctypes.byref(n),
                              None) == binding.RAG_ERR_INVALID_ARG


# ---- group-quantized int4-weight GEMM --------------------------------------
def _awq(**kw):
    a = dict(x=FAKE, qw=FAKE, s=FAKE, z=FAKE, y=FAKE, M=64, N=256, K=512, G=128, ws=FAKE,
             ws_bytes=1 << 30)
    a.update(kw)
    return binding.lib().rag_awq_gemm(a["x"], a["qw"], a["s"], a["z"], a["y"], a["M"], a["N"],
                                      a["K"], a["G"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), binding.RAG_ERR_INVALID_ARG),
    (dict(z=None), binding.RAG_ERR_INVALID_ARG),
    (dict(x=FAKE + 8), binding.RAG_ERR_INVALID_ARG),
    (dict(s=FAKE + 2), binding.RAG_ERR_INVALID_ARG),
    (dict(z=FAKE + 8), binding.RAG_ERR_INVALID_ARG),
    (dict(M=-1), binding.RAG_ERR_INVALID_ARG),
    (dict(N=0), binding.RAG_ERR_INVALID_ARG),
    (dict(G=64), binding.RAG_ERR_UNSUPPORTED),
    (dict(K=500), binding.RAG_ERR_UNSUPPORTED),
    (dict(N=200), binding.RAG_ERR_UNSUPPORTED),
    (dict(M=5_000_000), binding.RAG_ERR_UNSUPPORTED),
    (dict(ws=None), binding.RAG_ERR_WORKSPACE),
    (dict(ws_bytes=100, M=16, N=4096, K=14336), binding.RAG_ERR_WORKSPACE),
    (dict(ws=FAKE + 16), binding.RAG_ERR_INVALID_ARG),
    (dict(M=0, x=None, y=None, ws=None, ws_bytes=0), binding.RAG_OK),  # nothing to compute
    (dict(M=0, qw=None), binding.RAG_ERR_INVALID_ARG),
])
def test_awq_validation(kw, status):
    assert _awq(**kw) == status
    if status != binding.RAG_OK:
        assert binding.rag_last_error().startswith("awq gemm")


def test_awq_workspace_size():
    ws = binding.rag_awq_workspace_size
    assert ws(0, 256, 512) == 0
    assert ws(64, 256, 500) == 0 and ws(64, 256, 512, 64) == 0
    # enough tiles to fill the GPU: only the group-sum pieces, 16 bytes per
    # (group, row), 256-byte rounded
    M, N, K = 4096, 4096, 4096
    assert ws(M, N, K) == (K // 128) * M * 16
    # few 128-row output tiles: group sums plus a whole number of fp32
    # [M, N] partial planes of a split over the groups
    M, N, K = 200, 1024, 2048
    pieces = -(-(K // 128) * M * 16 // 256) * 256
    assert ws(M, N, K) > pieces and (ws(M, N, K) - pieces) % (M * N * 4) == 0
    # small batches (M <= 64): nothing when a workgroup's X fits its LDS
    # (qkv, o, gate_up of the 7B model at 16 rows); with the groups split over
    # workgroups, counters for at least N / 128 column blocks
    # (256-byte rounded) and whole fp32 [M, N] partial planes
    assert ws(16, 6144, 4096) == 0 and ws(16, 28672, 4096) == 0

    def split_parts(M, N, K):
        b = ws(M, N, K)
        counters = b % (M * N * 4)
        return b // (M * N * 4), counters
    # 112 groups of x (4 KB each per 16 rows) exceed a workgroup's 128 KB of
    # LDS: at least 4 splits
    s, c = split_parts(16, 4096, 14336)
    assert s >= 4 and c >= 4 * (4096 // 128) and c % 256 == 0
    s, c = split_parts(20, 4096, 14336)         # two row blocks: at least 7 splits
    assert s >= 7 and c >= 4 * (4096 // 128)
    assert ws(16, 4096, 4096) == 0              # 32 groups fit: no split


def test_awq_pack_layout():
    """Every code lands at the documented position: word 8a + 4b + c of
    (group g, column n) holds k = 128g + 8(4c + 2b + a) + j at bits
    4(j/2) + 16(j%2)."""
    r = np.random.Generator(np.random.PCG64(3))
    K, N = 384, 256
    q = r.integers(0, 16, size=(K, N), dtype=np.uint8)
    packed = binding.rag_awq_pack_weights(q).view(np.uint32)
    assert packed.shape == (K // 128, N, 16)
    back = np.zeros_like(q)
    for w in range(16):
        a, b, c = w >> 3, (w >> 2) & 1, w & 3
        for j in range(8):
            k = np.arange(K // 128) * 128 + 8 * (4 * c + 2 * b + a) + j
            back[k, :] = (packed[:, :, w] >> (4 * (j // 2) + 16 * (j % 2))) & 15
    assert np.array_equal(back, q)


def test_awq_pack_errors():
    q = np.zeros((256, 128), dtype=np.uint8)
    q[200, 5] = 16
    with pytest.raises(binding.RagError, match="not 4-bit"):
        binding.rag_awq_pack_weights(q)
    with pytest.raises(binding.RagError, match="group_size"):
        binding.rag_awq_pack_weights(np.zeros((256, 128), np.uint8), group_size=64)
    with pytest.raises(binding.RagError, match="multiple of 128"):
        binding.rag_awq_pack_weights(np.zeros((256, 100), np.uint8))
