"""GPU parity of the group-quantized int4-weight GEMM (rag_awq_gemm) against
the fp64 oracle (dequantize per group, then multiply).

Tolerance, from the arithmetic: the kernel's products are exact and its sums
run in fp32 over 128-term group sums, so its error before the final rounding
is at most about 128 * 2^-24 = 2^-17 times A = sum_k |x| (|q| + 128 + |z| +
128) |s| (the magnitudes entering those sums).  The large-batch kernel also
rescales its running sums once per group by a ratio of scale mantissas
(rounded, reciprocal within 1 ulp): at most G * 2^-22 times A more over G
groups.  y is then rounded to bf16 (half an ulp, 2^-9 relative).  Each
element must satisfy |y - ref| <= 2^-8 |ref| + (2^-17 + G 2^-22) A, and with
these inputs (outputs of order 1) the attention path's max-abs 2e-2 /
mean-abs 2e-3 bar as well.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2412_10543_amd import binding
from paper_2412_10543_amd.workloads import AWQ_LAYERS_7B, awq_problem

import gpu_support as G_

pytestmark = pytest.mark.gpu


def _device(p):
    qw = torch.from_numpy(binding.rag_awq_pack_weights(p.codes)).cuda()
    return qw, p.scales.cuda(), torch.from_numpy(p.zeros).cuda()


def _workspace(M, N, K):
    return torch.zeros(max(binding.rag_awq_workspace_size(M, N, K), 1), dtype=torch.uint8,
                       device="cuda")


def _run(p, qw, sc, z, ws=None):
    M, K = p.x.shape
    N = p.codes.shape[1]
    y = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    ws = _workspace(M, N, K) if ws is None else ws
    binding.rag_awq_gemm(p.x, qw, sc, z, y, ws)
    torch.cuda.synchronize()
    return y


def _check(p, y, rows=None, cols=None):
    x = p.x.float().cpu().numpy().astype(np.float64)
    s = p.scales.float().numpy().astype(np.float64)
    rows = np.arange(x.shape[0]) if rows is None else rows
    cols = np.arange(p.codes.shape[1]) if cols is None else cols
    xr = x[rows]
    ref = oracle.awq_gemm(xr, p.codes[:, cols], p.zeros[:, cols], s[:, cols], 128)
    g = np.arange(p.codes.shape[0]) // 128
    mag = (p.codes[:, cols].astype(np.float64) + p.zeros[g][:, cols] + 256) * s[g][:, cols]
    G = p.codes.shape[0] // 128
    bound = 2.0 ** -8 * np.abs(ref) + (2.0 ** -17 + G * 2.0 ** -22) * (np.abs(xr) @ mag)
    got = y.float().cpu().numpy().astype(np.float64)[np.ix_(rows, cols)]
    assert np.all(np.isfinite(got)), "non-finite output"
    err = np.abs(got - ref)
    worst = np.unravel_index(np.argmax(err - bound), err.shape)
    assert np.all(err <= bound), f"err {err[worst]:.3e} > bound {bound[worst]:.3e} at {worst}"
    if np.abs(ref).max() < 64:       # outputs of order 1 (not the scale-range case)
        G_.assert_parity(got, ref, "awq")


@pytest.mark.parametrize("M,N,K", [
    (1, 128, 128), (7, 256, 384), (64, 128, 256), (77, 384, 1024), (130, 512, 512),
    (16, 4096, 4096), (256, 1024, 2048), (333, 256, 14336 // 4), (1000, 640, 256),
    (5, 256, 8192), (40, 384, 10240), (20, 512, 1024)])
def test_awq_parity(M, N, K):
    p = awq_problem(M, N, K, seed=M * 7 + N + K, device="cuda")
    _check(p, _run(p, *_device(p)))


@pytest.mark.parametrize("name,K,N", AWQ_LAYERS_7B)
@pytest.mark.parametrize("M", [16, 40, 64, 8192])
def test_awq_7b_layers_sampled(name, K, N, M):
    """The 7B model's linear layers at decode batches (16 rows, the shape the
    bench times; 40 and 64 rows: 8-block column tiles on 2 or 4 waves) and a
    chunked-prefill batch; sampled rows and columns (first, last, random)
    against the oracle."""
    p = awq_problem(M, N, K, seed=K + N + M, device="cuda")
    y = _run(p, *_device(p))
    r = np.random.Generator(np.random.PCG64(M + N))
    rows = np.unique(np.concatenate([[0, M - 1], r.integers(0, M, 14)]))
    cols = np.unique(np.concatenate([[0, 127, 128, N - 1], r.integers(0, N, 60)]))
    _check(p, y, rows, cols)


def test_awq_deterministic_and_extremes():
    """Two runs give identical bits (fixed-order split reduction); codes and
    zero points at 0 and 15 and zero scales are handled exactly."""
    M, N, K = 24, 1024, 2048
    p = awq_problem(M, N, K, seed=5, device="cuda")
    p.codes[:128] = 15
    p.zeros[0] = 0
    p.codes[128:256] = 0
    p.zeros[1] = 15
    p.scales[2] = 0.0
    dev = _device(p)
    a, b = _run(p, *dev), _run(p, *dev)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    _check(p, a)


@pytest.mark.parametrize("M,N,K,nb,splits", [
    (16, 4096, 14336, None, None),    # 112 groups: split at least 4 ways (X staged in LDS)
    (16, 4096, 4096, None, 2),        # o_proj shape, split in two
    (3, 1024, 2048, 8, 3),            # 8 column blocks, uneven split (16 groups / 3)
    (3, 1024, 2048, 1, 3),            # one column block per workgroup, uneven split
    (40, 512, 4096, 2, 5),            # 3 row blocks (padded to 4), uneven split
    (64, 256, 1024, 2, 8),            # one group per workgroup
    (9, 1024, 2432, 8, 2),            # 8 blocks on 2 waves x 4 phases, uneven (3, 3, 3, 1)
    (32, 2048, 1024, 8, None),        # 2 row blocks, 8 blocks on 2 waves, no split
    (17, 1024, 3200, 8, 2),           # 2 row blocks (padded), phases of 4, 4, 4, 1 groups
    (50, 1024, 1536, 8, 3),           # 4 row blocks (padded), 8 blocks on 4 waves x 2 phases
    (64, 512, 2048, 4, None)])        # 4 row blocks, 4 blocks on 2 waves x 4 phases
def test_awq_small_batch_splits_reuse_workspace(M, N, K, nb, splits):
    """Small batches split over the weight groups: the last workgroup of a
    column block adds the fp32 partials and resets its arrival counter, so one
    workspace, zero-filled once, serves every later call (three calls, fresh
    inputs each time), and a repeat gives identical bits.  The column blocks
    of a workgroup are shared by 1, 2 or 4 waves, each taking a range of the
    groups (phases of uneven length included)."""
    with G_.env("RAG_AWQ_SM_NB", nb), G_.env("RAG_AWQ_SM_SPLITS", splits):
        ws = _workspace(M, N, K)
        first = None
        for call in range(3):
            p = awq_problem(M, N, K, seed=M + N + K + call, device="cuda")
            dev = _device(p)
            y = _run(p, *dev, ws=ws)
            _check(p, y)
            if call == 0:
                first = (p, dev, y)
        p, dev, y = first
        assert torch.equal(_run(p, *dev, ws=ws).view(torch.int16), y.view(torch.int16))
        # with a split, the counters (one per column block, at least N / 128
        # of them) are zero again
        if binding.rag_awq_workspace_size(M, N, K) > 0:
            assert int(ws[:4 * (N // 128)].count_nonzero()) == 0
        else:
            assert splits is None and M * (K // 128) <= 32 * 16


@pytest.mark.parametrize("M,N", [(130, 512), (20, 256)])
def test_awq_scale_range(M, N):
    """Scales across the bf16 range, per group: zero, subnormal (2^-130),
    2^-126 * 1.5, 2^-60, 2^60, negative, and a mix per column; on the large
    (LDS-staged) and the small-batch path."""
    K = 1024
    p = awq_problem(M, N, K, seed=M + N, device="cuda")
    vals = [0.0, 2.0 ** -130, 1.5 * 2.0 ** -126, 2.0 ** -60, 2.0 ** 60, -0.02, 3e-3]
    s = p.scales.float()
    for g, v in enumerate(vals):
        s[g] = v
    r = np.random.Generator(np.random.PCG64(M))
    s[7] = torch.from_numpy(np.array(vals)[r.integers(0, len(vals), N)].astype(np.float32))
    p.scales = s.to(torch.bfloat16)
    _check(p, _run(p, *_device(p)))


def test_awq_zero_weights():
    """q == z everywhere: every weight is zero; y is zero up to the fp32
    cancellation between the code sums and the zero-point term (the bound's
    2^-17 A part, as ref is 0)."""
    M, N, K = 40, 256, 512
    p = awq_problem(M, N, K, seed=9, device="cuda")
    p.codes[:] = 6
    p.zeros[:] = 6
    _check(p, _run(p, *_device(p)))


def test_awq_empty_batch():
    p = awq_problem(0, 256, 256, seed=1, device="cuda")
    qw, sc, z = _device(p)
    y = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    binding.rag_awq_gemm(p.x, qw, sc, z, y, None)
    torch.cuda.synchronize()


@pytest.mark.parametrize("seed", [3, 4])
def test_awq_random_shapes(seed):
    """Seeded random shapes on both kernels: M 1-300, N and K multiples of
    128 up to 2048 and 5120 (small batches split or not, large batches with and
    without the group split)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    for case in range(12):
        M = int(rng.integers(1, 301))
        N = 128 * int(rng.integers(1, 17))
        K = 128 * int(rng.integers(1, 41))
        p = awq_problem(M, N, K, seed=seed * 1000 + case, device="cuda")
        _check(p, _run(p, *_device(p)))
