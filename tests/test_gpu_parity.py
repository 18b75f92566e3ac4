"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle on
small seeded inputs that still span several tiles and ragged tails, plus the
invariants the GPU path must keep.  Tolerance: max-abs 2e-2, mean-abs 2e-3."""
import numpy as np
import pytest
import torch

import gpu_support as G
from paper_2412_10543_amd import binding
from paper_2412_10543_amd.workloads import normal_bf16, paged_pool

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------------------
# prefill
# ---------------------------------------------------------------------------
PREFILL_LENS = [[1], [2], [15], [16], [17], [63], [64], [65], [127], [128], [129], [300],
                [1, 129, 64, 333, 7], [0, 5, 0, 200]]


@pytest.mark.parametrize("lens", PREFILL_LENS, ids=lambda x: "-".join(map(str, x)))
@pytest.mark.parametrize("hq,hkv,d", [(4, 2, 64), (8, 8, 128), (8, 1, 128), (32, 8, 128)])
def test_prefill_causal(orc, lens, hq, hkv, d):
    q, k, v = G.prefill_inputs(lens, lens, hq, hkv, d, seed=sum(lens) + hq + d)
    sc = G.scale_for(d)
    o, lse = G.gpu_prefill(q, k, v, lens, lens, sc)
    ro, rl = G.oracle_prefill(orc, q, k, v, lens, lens, sc)
    G.assert_parity(o, ro, "prefill o")
    got = lse.cpu().numpy()
    assert np.max(np.abs(got - rl)) < 1e-3, "lse"


@pytest.mark.parametrize("lens", [[1], [70], [129, 3]], ids=str)
@pytest.mark.parametrize("d", [64, 128])
def test_prefill_noncausal(orc, lens, d):
    q, k, v = G.prefill_inputs(lens, lens, 8, 2, d, seed=77 + d)
    o, lse = G.gpu_prefill(q, k, v, lens, lens, G.scale_for(d), causal=False)
    ro, rl = G.oracle_prefill(orc, q, k, v, lens, lens, G.scale_for(d), causal=False)
    G.assert_parity(o, ro, "non-causal")


def test_prefill_suffix_rows(orc):
    """Fewer query rows than keys (a chunk of a longer prompt): bottom-right
    causal alignment."""
    lq, lk = [1, 40, 130, 64], [1, 300, 131, 640]
    q, k, v = G.prefill_inputs(lq, lk, 8, 2, 128, seed=5)
    o, _ = G.gpu_prefill(q, k, v, lq, lk, G.scale_for(128))
    ro, _ = G.oracle_prefill(orc, q, k, v, lq, lk, G.scale_for(128))
    G.assert_parity(o, ro, "suffix")


@pytest.mark.parametrize("q_scale", [4.0, 8.0])
def test_prefill_peaky_scores(orc, q_scale):
    """Large scores exercise the running-maximum rescaling."""
    lens = [300, 77]
    q, k, v = G.prefill_inputs(lens, lens, 8, 2, 128, seed=9, q_scale=q_scale)
    o, lse = G.gpu_prefill(q, k, v, lens, lens, G.scale_for(128))
    ro, rl = G.oracle_prefill(orc, q, k, v, lens, lens, G.scale_for(128))
    G.assert_parity(o, ro, "peaky")
    assert np.max(np.abs(lse.cpu().numpy() - rl)) < 2e-2


def test_prefill_repeatable_and_packing_order(orc):
    lens = [200, 17, 129, 64]
    q, k, v = G.prefill_inputs(lens, lens, 8, 2, 128, seed=12)
    o1, l1 = G.gpu_prefill(q, k, v, lens, lens, G.scale_for(128))
    o2, l2 = G.gpu_prefill(q, k, v, lens, lens, G.scale_for(128))
    assert torch.equal(o1, o2) and torch.equal(l1, l2), "run-to-run bitwise"
    cu = G.cu_from_lens(lens)
    order = [2, 0, 3, 1]
    idx = torch.cat([torch.arange(cu[s], cu[s + 1]) for s in order]).cuda()
    lens2 = [lens[s] for s in order]
    o3, l3 = G.gpu_prefill(q[idx].contiguous(), k[idx].contiguous(), v[idx].contiguous(),
                           lens2, lens2, G.scale_for(128))
    assert torch.equal(o3, o1[idx]), "packing order, bitwise"


# ---------------------------------------------------------------------------
# paged decode
# ---------------------------------------------------------------------------
DECODE_LENS = [[1], [15], [16], [17], [33], [1000], [1, 17, 500, 2049, 64]]


@pytest.mark.parametrize("kv_lens", DECODE_LENS, ids=lambda x: "-".join(map(str, x)))
@pytest.mark.parametrize("hq,hkv,d", [(4, 2, 64), (32, 8, 128), (8, 8, 128), (16, 1, 128)])
@pytest.mark.parametrize("splits", [1, 0, 3])
def test_decode(orc, kv_lens, hq, hkv, d, splits):
    q, pool = G.decode_case(kv_lens, hq, hkv, d, seed=len(kv_lens) * 31 + hq)
    o = G.gpu_paged(q, pool, hq, hkv, d, G.scale_for(d), num_splits=splits)
    ro = G.oracle_paged(orc, q, pool, G.scale_for(d))
    G.assert_parity(o, ro, f"decode splits={splits}")


@pytest.mark.parametrize("seed", [1, 2])
def test_decode_balanced_units_many_rows(orc, seed):
    """Automatic policy with fewer (row, kv head) pairs than CUs: units cut
    the pages of all rows into equal ranges, so one unit covers pieces of
    several short rows and long rows span several units.  Against the oracle
    and within rounding of a uniform two-way split."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = [int(x) for x in rng.integers(1, 3000, size=28)] + [9000, 1]   # 30 x 8 pairs < 256
    q, pool = G.decode_case(lens, 32, 8, 128, seed=seed + 40)
    o = G.gpu_paged(q, pool, 32, 8, 128, G.scale_for(128), num_splits=0)
    G.assert_parity(o, G.oracle_paged(orc, q, pool, G.scale_for(128)), "balanced")
    o2 = G.gpu_paged(q, pool, 32, 8, 128, G.scale_for(128), num_splits=2)
    assert float((o.float() - o2.float()).abs().max()) < 1e-2


@pytest.mark.parametrize("n_rows,hq,hkv", [(100, 16, 2), (200, 8, 1), (255, 4, 1)])
def test_decode_balanced_units_rows_past_64(orc, n_rows, hq, hkv):
    """Balanced units (fewer (row, kv head) pairs than CUs) with more than 64
    rows: each unit reads the lengths in chunks of 64 rows (up to four) and
    walks all of them; lengths from 1 to 800 with a few long rows."""
    rng = np.random.Generator(np.random.PCG64(n_rows + hq))
    lens = [int(x) for x in rng.integers(1, 800, size=n_rows)]
    for i in (0, n_rows // 2, n_rows - 1):
        lens[i] = 4000 + i
    q, pool = G.decode_case(lens, hq, hkv, 128, seed=n_rows * 3 + hkv)
    o = G.gpu_paged(q, pool, hq, hkv, 128, G.scale_for(128), num_splits=0)
    G.assert_parity(o, G.oracle_paged(orc, q, pool, G.scale_for(128)), "balanced, rows past 64")


def test_decode_split_merge_repeatable(orc):
    """The in-kernel split merge relies on completed device-coherent stores
    and a device-scope arrival count: 64 calls with 16 splits (and with the
    automatic policy) must give bit-identical outputs, and the result the
    oracle's."""
    q, pool = G.decode_case([4000, 900, 7000, 33], 32, 8, 128, seed=77)
    for splits in (16, 0):
        ws = G.workspace_for(4, 32, 8, 128, pool.block_tables.shape[1], splits)
        kl = G.to_dev_i32(pool.kv_lens)
        outs = []
        for _ in range(64):
            o = torch.empty_like(q)
            binding.rag_attn_decode_paged(q, pool.k_cache, pool.v_cache, o, pool.block_tables, kl,
                                          G.scale_for(128), num_splits=splits, workspace=ws)
            outs.append(o)
        torch.cuda.synchronize()
        for o in outs[1:]:
            assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16)), splits
        G.assert_parity(outs[0], G.oracle_paged(orc, q, pool, G.scale_for(128)), f"splits {splits}")


def test_decode_peaky(orc):
    q, pool = G.decode_case([700, 33, 4000], 32, 8, 128, seed=3, q_scale=8.0)
    o = G.gpu_paged(q, pool, 32, 8, 128, G.scale_for(128))
    G.assert_parity(o, G.oracle_paged(orc, q, pool, G.scale_for(128)), "decode peaky")


def test_decode_page_permutation_and_repeatability():
    kv = [300, 45, 1024, 7]
    q, pool = G.decode_case(kv, 32, 8, 128, seed=21)
    o1 = G.gpu_paged(q, pool, 32, 8, 128, G.scale_for(128))
    o2 = G.gpu_paged(q, pool, 32, 8, 128, G.scale_for(128))
    assert torch.equal(o1, o2), "run-to-run bitwise"
    perm = torch.randperm(pool.num_blocks, generator=torch.Generator().manual_seed(5)).cuda()
    inv = torch.argsort(perm)
    moved = paged_pool(kv, 8, 128, 21, device="cuda")
    moved.k_cache = pool.k_cache[inv].contiguous()
    moved.v_cache = pool.v_cache[inv].contiguous()
    moved.block_tables = perm[pool.block_tables.long()].to(torch.int32).contiguous()
    o3 = G.gpu_paged(q, moved, 32, 8, 128, G.scale_for(128))
    assert torch.equal(o1, o3), "physical page order, bitwise"


def test_decode_matches_prefill_last_row():
    """Paged decode over L keys equals the last row of a dense causal prefill
    over the same L tokens (two different kernels, within tolerance)."""
    L, hq, hkv, d = 777, 32, 8, 128
    q, pool = G.decode_case([L], hq, hkv, d, seed=8)
    nb = (L + 15) // 16
    blocks = pool.block_tables[0, :nb].long()
    kd = pool.k_cache[blocks].permute(0, 2, 1, 3).reshape(nb * 16, hkv, d)[:L].contiguous()
    vd = pool.v_cache[blocks].permute(0, 2, 1, 3).reshape(nb * 16, hkv, d)[:L].contiguous()
    qd = normal_bf16((L, hq, d), 99, "cuda")
    qd[L - 1] = q[0]
    o_pf, _ = G.gpu_prefill(qd, kd, vd, [L], [L], G.scale_for(d))
    o_dec = G.gpu_paged(q, pool, hq, hkv, d, G.scale_for(d))
    mx, mean = G.errors(o_dec[0], o_pf[L - 1].float().cpu().numpy())
    assert mx <= 2 * G.MAX_ABS and mean <= 2 * G.MEAN_ABS


def test_decode_workspace_left_zeroed(orc):
    """The in-kernel split merge counts arrivals in the workspace; every call
    must leave the counters at zero, so back-to-back calls stay correct."""
    q, pool = G.decode_case([3000, 70, 1500], 32, 8, 128, seed=41)
    ws = G.workspace_for(3, 32, 8, 128, pool.block_tables.shape[1], num_splits=6)
    ro = G.oracle_paged(orc, q, pool, G.scale_for(128))
    outs = []
    for _ in range(3):
        o = torch.empty_like(q)
        from paper_2412_10543_amd import binding
        binding.rag_attn_decode_paged(q, pool.k_cache, pool.v_cache, o, pool.block_tables,
                                      G.to_dev_i32(pool.kv_lens), G.scale_for(128),
                                      num_splits=6, workspace=ws)
        torch.cuda.synchronize()
        assert int(ws[:3 * 8 * 4].count_nonzero()) == 0, "arrival counters not reset"
        G.assert_parity(o, ro, "repeated split call")
        outs.append(o)
    assert torch.equal(outs[0], outs[1]) and torch.equal(outs[1], outs[2])


@pytest.mark.parametrize("n_rows,hq,hkv,splits", [(300, 32, 8, 0), (300, 32, 8, 2),
                                                  (1100, 8, 1, 4), (60, 8, 8, 0)])
def test_decode_uneven_rows(orc, n_rows, hq, hkv, splits):
    """Many rows of very different length in one batch: one long row among
    hundreds of short ones, so most splits of the short rows are empty while
    the long row uses all of them."""
    rng = np.random.Generator(np.random.PCG64(n_rows * 7 + splits))
    kv = [int(x) for x in rng.integers(1, 400, size=n_rows)]
    kv[n_rows // 3] = 5000
    q, pool = G.decode_case(kv, hq, hkv, 128, seed=n_rows + hq)
    o = G.gpu_paged(q, pool, hq, hkv, 128, G.scale_for(128), num_splits=splits)
    G.assert_parity(o, G.oracle_paged(orc, q, pool, G.scale_for(128)), "balanced decode")


def test_decode_one_row_max_pieces(orc):
    """A single long row on one kv head is cut into close to the maximum of 64
    splits, all merged in the kernel."""
    q, pool = G.decode_case([20000], 4, 1, 128, seed=31)
    from paper_2412_10543_amd import binding
    assert binding.rag_attn_decode_num_splits(1, 1, pool.block_tables.shape[1]) >= 60
    o = G.gpu_paged(q, pool, 4, 1, 128, G.scale_for(128))
    G.assert_parity(o, G.oracle_paged(orc, q, pool, G.scale_for(128)), "64 pieces")


def test_decode_splits_agree():
    q, pool = G.decode_case([5000, 3000], 32, 8, 128, seed=4)
    o1 = G.gpu_paged(q, pool, 32, 8, 128, G.scale_for(128), num_splits=1)
    o8 = G.gpu_paged(q, pool, 32, 8, 128, G.scale_for(128), num_splits=8)
    mx, mean = G.errors(o8, o1.float().cpu().numpy())
    assert mx <= G.MAX_ABS and mean <= G.MEAN_ABS


# ---------------------------------------------------------------------------
# mixed decode + chunked prefill in one launch
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("d,hq,hkv", [(128, 32, 8), (64, 4, 2)])
def test_mixed_batch(orc, d, hq, hkv):
    dec_kv = [100, 17, 3000, 1]
    pieces = [(1, 0), (300, 500), (129, 129), (64, 1000)]   # (q_len, prior context)
    kv = dec_kv + [nq + p for nq, p in pieces]
    pool = paged_pool(kv, hkv, d, 17, device="cuda")
    q_lens = [1] * len(dec_kv) + [nq for nq, _ in pieces]
    cu = G.cu_from_lens(q_lens)
    q = normal_bf16((cu[-1], hq, d), 18, "cuda")
    o = G.gpu_paged(q, pool, hq, hkv, d, G.scale_for(d), cu_q=cu, num_decode=len(dec_kv),
                    max_seqlen_q=max(q_lens))
    ro = G.oracle_paged(orc, q, pool, G.scale_for(d), cu_q=cu)
    G.assert_parity(o, ro, "mixed")


def test_mixed_empty_piece_and_pieces_only(orc):
    kv = [40, 500, 260]
    q_lens = [0, 200, 260]
    pool = paged_pool(kv, 8, 128, 23, device="cuda")
    cu = G.cu_from_lens(q_lens)
    q = normal_bf16((cu[-1], 32, 128), 24, "cuda")
    o = G.gpu_paged(q, pool, 32, 8, 128, G.scale_for(128), cu_q=cu, num_decode=0,
                    max_seqlen_q=260)
    G.assert_parity(o, G.oracle_paged(orc, q, pool, G.scale_for(128), cu_q=cu), "pieces")
