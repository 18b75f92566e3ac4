"""The measurement probes of bench.py --ceilings run on small inputs: every
entry point launches and returns 0, the memory probes with both load policies
and all K/V page patterns (each load of a probe stays inside its buffers: page
ids index whole pages of the pool, the stream read stops at its length), and
bad arguments are rejected before any launch."""
import ctypes

import pytest
import torch

from paper_2412_10543_amd import build as pb

pytestmark = pytest.mark.gpu

vp = ctypes.c_void_p


def _lib():
    L = ctypes.CDLL(pb.PROBES)
    L.rag_probe_page_read.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                      vp, vp]
    L.rag_probe_kv_page_read.argtypes = [vp, vp, vp, ctypes.c_int64, ctypes.c_int32,
                                         ctypes.c_int32, vp, vp]
    L.rag_probe_stream_read.argtypes = [vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, vp,
                                        vp]
    for n in ("rag_probe_mfma_loop", "rag_probe_attn_slot", "rag_probe_softmax_mfma",
              "rag_probe_attn_pair"):
        getattr(L, n).argtypes = [ctypes.c_int32, ctypes.c_int32, vp, vp]
    return L


def test_probes_launch_small():
    L = _lib()
    s = torch.cuda.current_stream().cuda_stream
    pages = 4096                                        # 16 MiB pool of 4 KB pages
    pool = torch.full((pages * 1024,), 7, dtype=torch.int32, device="cuda")
    pool2 = torch.full((pages * 1024,), 9, dtype=torch.int32, device="cuda")
    ids = torch.randperm(pages, generator=torch.Generator().manual_seed(3))[:1000]
    ids = ids.to(torch.int32).cuda()
    sink = torch.zeros(1 << 16, dtype=torch.int32, device="cuda")
    for hint in (0, 1):
        assert L.rag_probe_page_read(pool.data_ptr(), ids.data_ptr(), 1000, 64, hint,
                                     sink.data_ptr(), s) == 0
        assert L.rag_probe_stream_read(pool.data_ptr(), pool.numel() * 4 - 48, 64, hint,
                                       sink.data_ptr(), s) == 0
    for pattern in (0, 1, 2):
        assert L.rag_probe_kv_page_read(pool.data_ptr(), pool2.data_ptr(), ids.data_ptr(), 999,
                                        64, pattern, sink.data_ptr(), s) == 0
    for n in ("rag_probe_mfma_loop", "rag_probe_attn_slot", "rag_probe_softmax_mfma",
              "rag_probe_attn_pair"):
        assert getattr(L, n)(3, 8, sink.data_ptr(), s) == 0
    torch.cuda.synchronize()
    # rejected before a launch
    assert L.rag_probe_kv_page_read(pool.data_ptr(), pool2.data_ptr(), ids.data_ptr(), 10, 64, 3,
                                    sink.data_ptr(), s) == -1
    assert L.rag_probe_kv_page_read(None, pool2.data_ptr(), ids.data_ptr(), 10, 64, 0,
                                    sink.data_ptr(), s) == -1
    assert L.rag_probe_stream_read(pool.data_ptr(), -16, 64, 0, sink.data_ptr(), s) == -1
    assert L.rag_probe_page_read(pool.data_ptr(), ids.data_ptr(), 10, 0, 0, sink.data_ptr(),
                                 s) == -1
