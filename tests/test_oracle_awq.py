"""Pins of the oracle's int4-weight GEMM (oracle/awq.py), on the CPU:
brute force, special cases with exact answers, group structure, and planted
mistakes the pins must catch."""
import numpy as np
import pytest

from oracle import awq_gemm, dequantize
from oracle.attention import bf16_bits_to_f64


def _case(M, K, N, G, seed):
    r = np.random.Generator(np.random.PCG64(seed))
    x = r.standard_normal((M, K))
    q = r.integers(0, 16, size=(K, N))
    z = r.integers(0, 16, size=(K // G, N))
    s = r.uniform(0.001, 0.05, size=(K // G, N))
    return x, q, z, s


def _brute(x, q, z, s, G):
    M, K = x.shape
    N = q.shape[1]
    y = np.zeros((M, N))
    for m in range(M):
        for n in range(N):
            acc = 0.0
            for k in range(K):
                acc += x[m, k] * (q[k, n] - z[k // G, n]) * s[k // G, n]
            y[m, n] = acc
    return y


@pytest.mark.parametrize("M,K,N,G", [(1, 8, 3, 4), (3, 16, 5, 8), (4, 32, 2, 16)])
def test_brute_force(M, K, N, G):
    x, q, z, s = _case(M, K, N, G, M * K + N)
    assert np.allclose(awq_gemm(x, q, z, s, G), _brute(x, q, z, s, G), rtol=1e-12, atol=1e-12)


def test_codes_at_zero_point_give_zero():
    x, q, z, s = _case(5, 64, 7, 32, 1)
    q = np.repeat(z, 32, axis=0)
    assert np.array_equal(awq_gemm(x, q, z, s, 32), np.zeros((5, 7)))


def test_unit_scales_zero_points_are_integer_matmul():
    r = np.random.Generator(np.random.PCG64(2))
    x = r.integers(-8, 9, size=(6, 64))
    q = r.integers(0, 16, size=(64, 9))
    z = np.zeros((2, 9), dtype=np.int64)
    s = np.ones((2, 9))
    assert np.array_equal(awq_gemm(x, q, z, s, 32), (x @ q).astype(np.float64))


def test_group_structure():
    """Scaling group g's scales by a scales exactly the contribution of rows
    k in group g; other groups are untouched."""
    x, q, z, s = _case(4, 96, 5, 32, 3)
    y = awq_gemm(x, q, z, s, 32)
    s2 = s.copy()
    s2[1] *= 3.0
    y2 = awq_gemm(x, q, z, s2, 32)
    part = x[:, 32:64] @ ((q[32:64] - z[1]) * s[1])
    assert np.allclose(y2 - y, 2.0 * part, rtol=1e-12, atol=1e-12)


def test_bf16_scales_widened_exactly():
    s_bits = np.array([[0x3F80, 0x3E00]], dtype=np.uint16)       # 1.0, 0.125
    assert np.array_equal(bf16_bits_to_f64(s_bits), np.array([[1.0, 0.125]]))
    W = dequantize(np.array([[3, 5]]), np.array([[1, 1]]), s_bits, 1)
    assert np.array_equal(W, np.array([[2.0, 0.5]]))


def _mutant_zero_added(x, q, z, s, G):
    g = np.arange(q.shape[0]) // G
    return x @ ((q + z[g]) * s[g])


def _mutant_last_group_scale(x, q, z, s, G):
    g = np.minimum(np.arange(q.shape[0]) // G + 1, z.shape[0] - 1)
    return x @ ((q - z[g]) * s[g])


def _mutant_scale_by_k(x, q, z, s, G):
    g = np.arange(q.shape[0]) // G
    gk = np.arange(q.shape[0]) % z.shape[0]          # scale row picked by k, not by group
    return x @ ((q - z[g]) * s[gk])


def _mutant_codes_reversed_in_group(x, q, z, s, G):
    k = np.arange(q.shape[0])
    src = (k // G) * G + (G - 1 - k % G)              # an unpacking that reverses a group
    g = k // G
    return x @ ((q[src] - z[g]) * s[g])


@pytest.mark.parametrize("mutant", [_mutant_zero_added, _mutant_last_group_scale,
                                    _mutant_scale_by_k, _mutant_codes_reversed_in_group])
def test_planted_mistakes_are_caught(mutant):
    x, q, z, s = _case(3, 64, 4, 16, 9)
    assert not np.allclose(mutant(x, q, z, s, 16), _brute(x, q, z, s, 16))
