"""ctypes wrapper around the fp64 C oracle (``attn_oracle.c``).

Test infrastructure: only the tests, ``__graft_entry__.smoke()`` and the
bench's CPU-baseline leg may import this module.  It never imports the GPU
package and the GPU package never imports it.

Inputs arrive as bf16 bit patterns (``numpy.uint16``) or as float arrays; bf16
is widened to fp64 exactly (a bf16 value is the upper half of an IEEE fp32
word).  Outputs are fp64.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "attn_oracle.c")
LIBRARY = os.path.join(_HERE, "liboracle_attn.so")

_i32p = ctypes.POINTER(ctypes.c_int32)
_f64p = ctypes.POINTER(ctypes.c_double)


def build(source: str = SOURCE, out: str = LIBRARY) -> str:
    """Compile the oracle with gcc (OpenMP, -O2, no fast-math)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11", "-o", out,
           source, "-lm"]
    subprocess.run(cmd, check=True)
    return out


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to fp64."""
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16))
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _f64(x) -> np.ndarray:
    a = np.asarray(x)
    if a.dtype == np.uint16:
        return bf16_bits_to_f64(a)
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x), dtype=np.int32)


def _p(a: Optional[np.ndarray], t):
    if a is None:
        return ctypes.cast(None, t)
    return a.ctypes.data_as(t)


class Oracle:
    """Handle on one compiled oracle library (the shipped one, or a copy a
    test compiled from edited source)."""

    def __init__(self, path: str = LIBRARY):
        if path == LIBRARY and not os.path.exists(path):
            build()
        self.path = path
        lib = ctypes.CDLL(path)
        lib.oracle_attend_row.argtypes = [
            _f64p, ctypes.POINTER(_f64p), ctypes.POINTER(_f64p), ctypes.c_int32,
            ctypes.c_int32, ctypes.c_double, _f64p, _f64p, _f64p]
        lib.oracle_attention_varlen.argtypes = [
            _f64p, _f64p, _f64p, _f64p, _f64p, _i32p, _i32p, ctypes.c_int32,
            ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_double,
            ctypes.c_int32]
        lib.oracle_attention_paged.argtypes = [
            _f64p, _f64p, _f64p, _f64p, _f64p, _i32p, _i32p, _i32p,
            ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
            ctypes.c_int32, ctypes.c_int32, ctypes.c_double]
        lib.oracle_attention_seq_rows.argtypes = [
            _f64p, _f64p, _f64p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
            ctypes.c_int32, ctypes.c_int32, ctypes.c_double, ctypes.c_int32,
            _i32p, _i32p, ctypes.c_int32, _f64p, _f64p]
        for f in (lib.oracle_attend_row, lib.oracle_attention_varlen,
                  lib.oracle_attention_paged, lib.oracle_attention_seq_rows):
            f.restype = None
        self.lib = lib

    # -- one row -----------------------------------------------------------
    def attend_row(self, q, k_rows, v_rows, scale):
        """q [d]; k_rows, v_rows [n, d] (the visible keys in order).
        Returns (o [d], lse, p [n])."""
        q = _f64(q)
        k = _f64(k_rows)
        v = _f64(v_rows)
        n, d = k.shape
        kp = (_f64p * max(n, 1))(*[k[j].ctypes.data_as(_f64p) for j in range(n)])
        vp = (_f64p * max(n, 1))(*[v[j].ctypes.data_as(_f64p) for j in range(n)])
        o = np.zeros(d)
        lse = np.zeros(1)
        p = np.zeros(max(n, 1))
        self.lib.oracle_attend_row(_p(q, _f64p), kp, vp, n, d, float(scale),
                                   _p(o, _f64p), _p(lse, _f64p), _p(p, _f64p))
        return o, float(lse[0]), p[:n]

    # -- packed varlen ------------------------------------------------------
    def varlen(self, q, k, v, cu_q, cu_k, scale, causal=True, want_lse=True):
        """q [Tq, hq, d]; k, v [Tk, hkv, d]; cu_q, cu_k [S+1].
        Returns (o [Tq, hq, d], lse [hq, Tq] or None)."""
        q, k, v = _f64(q), _f64(k), _f64(v)
        cu_q, cu_k = _i32(cu_q), _i32(cu_k)
        tq, hq, d = q.shape
        hkv = k.shape[1]
        o = np.zeros_like(q)
        lse = np.zeros((hq, tq)) if want_lse else None
        self.lib.oracle_attention_varlen(
            _p(q, _f64p), _p(k, _f64p), _p(v, _f64p), _p(o, _f64p),
            _p(lse, _f64p), _p(cu_q, _i32p), _p(cu_k, _i32p), len(cu_q) - 1,
            hq, hkv, d, float(scale), int(bool(causal)))
        return o, lse

    # -- paged KV -------------------------------------------------------------
    def paged(self, q, k_cache, v_cache, block_tables, kv_lens, scale,
              cu_q=None, want_lse=True):
        """q [Tq, hq, d]; caches [num_blocks, hkv, bs, d];
        block_tables [S, max_blocks]; kv_lens [S]; cu_q [S+1] or None (one
        query row per sequence).  Returns (o, lse [hq, Tq] or None)."""
        q, kc, vc = _f64(q), _f64(k_cache), _f64(v_cache)
        bt, kl = _i32(block_tables), _i32(kv_lens)
        cq = None if cu_q is None else _i32(cu_q)
        tq, hq, d = q.shape
        _, hkv, bs, _ = kc.shape
        num_seqs, max_blocks = bt.shape
        o = np.zeros_like(q)
        lse = np.zeros((hq, tq)) if want_lse else None
        self.lib.oracle_attention_paged(
            _p(q, _f64p), _p(kc, _f64p), _p(vc, _f64p), _p(o, _f64p),
            _p(lse, _f64p), _p(bt, _i32p), _p(kl, _i32p), _p(cq, _i32p),
            num_seqs, max_blocks, bs, hq, hkv, d, float(scale))
        return o, lse

    # -- sampled rows of one sequence -----------------------------------------
    def seq_rows(self, q_rows, k, v, nq, row_idx, heads, hq, scale, causal=True):
        """q_rows [n, d]; k, v [nk, hkv, d] of one sequence; row_idx, heads [n].
        Returns (o_rows [n, d], lse_rows [n])."""
        qr, k, v = _f64(q_rows), _f64(k), _f64(v)
        ri, hd = _i32(row_idx), _i32(heads)
        n, d = qr.shape
        nk, hkv, _ = k.shape
        o = np.zeros((n, d))
        lse = np.zeros(n)
        self.lib.oracle_attention_seq_rows(
            _p(qr, _f64p), _p(k, _f64p), _p(v, _f64p), int(nq), nk, int(hq), hkv,
            d, float(scale), int(bool(causal)), _p(ri, _i32p), _p(hd, _i32p), n,
            _p(o, _f64p), _p(lse, _f64p))
        return o, lse


_default: Optional[Oracle] = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default
