"""Group-quantized int4-weight GEMM, written out from its definition.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``).

The served models are AWQ-quantized (Sec. "Setup"): every weight matrix W
[K, N] of the projections and the MLP is stored as 4-bit codes q in 0..15 with,
for each group of G consecutive input rows (k) and each output column n, a
zero point z and a scale s:

    W[k, n] = (q[k, n] - z[k // G, n]) * s[k // G, n]

and a layer computes Y = X W for activations X [M, K].  The oracle dequantizes
in fp64 and multiplies; bf16 inputs are widened exactly.
"""
from __future__ import annotations

import numpy as np

from .attention import bf16_bits_to_f64


def _f64(a):
    a = np.asarray(a)
    return bf16_bits_to_f64(a) if a.dtype == np.uint16 else a.astype(np.float64)


def dequantize(q, zeros, scales, group_size: int):
    """W [K, N] in fp64 from codes q [K, N], zeros [K/G, N], scales [K/G, N]."""
    q = np.asarray(q).astype(np.float64)
    z = np.asarray(zeros).astype(np.float64)
    s = _f64(scales)
    g = np.arange(q.shape[0]) // group_size
    return (q - z[g]) * s[g]


def awq_gemm(x, q, zeros, scales, group_size: int):
    """Y [M, N] = X [M, K] @ dequantize(...), fp64."""
    return _f64(x) @ dequantize(q, zeros, scales, group_size)
