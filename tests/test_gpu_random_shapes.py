"""GPU parity on seeded random shapes against the fp64 oracle: packed
prefill (causal or not, as many keys as queries or more, 0-5 query tiles per
workgroup forced), paged decode (automatic or explicit splits, up to 260 rows)
and mixed decode + chunked-prefill batches, over seven head shapes.  Each case
is drawn from a seeded generator, so a failure names a reproducible case."""
import numpy as np
import pytest

import gpu_support as G

pytestmark = pytest.mark.gpu

HEADS = [(4, 2, 64), (8, 8, 128), (8, 1, 128), (32, 8, 128), (16, 2, 64), (12, 4, 128),
         (64, 8, 128)]


def _case(orc, rng, case):
    hq, hkv, d = HEADS[rng.integers(len(HEADS))]
    kind = ["prefill", "prefill_k", "decode", "mixed"][rng.integers(4)]
    sc = G.scale_for(d)
    what = f"case {case}: {kind}, heads {hq}/{hkv}, d {d}"
    if kind.startswith("prefill"):
        n = int(rng.integers(1, 6))
        lq = [int(x) for x in rng.integers(0, 1500, size=n)]
        if max(lq) == 0:
            lq[0] = 1
        lk = [x + int(rng.integers(0, 300)) for x in lq] if kind == "prefill_k" else list(lq)
        causal = bool(rng.integers(2))
        items = int(rng.choice([0, 1, 2, 3, 5]))
        q, k, v = G.prefill_inputs(lq, lk, hq, hkv, d, seed=case * 13 + 1)
        with G.env("RAG_ATTN_PF_ITEMS", items if items else None):
            o, _ = G.gpu_prefill(q, k, v, lq, lk, sc, causal=causal)
        ro, _ = G.oracle_prefill(orc, q, k, v, lq, lk, sc, causal=causal)
        G.assert_parity(o, ro, f"{what}, q {lq}, k {lk}, causal {causal}, items {items}")
    elif kind == "decode":
        n = int(rng.integers(1, 260))
        kv = [int(x) for x in rng.integers(1, 3000, size=n)]
        splits = int(rng.choice([0, 0, 1, 2, 5, 17]))
        q, pool = G.decode_case(kv, hq, hkv, d, seed=case * 7 + 3)
        o = G.gpu_paged(q, pool, hq, hkv, d, sc, num_splits=splits)
        G.assert_parity(o, G.oracle_paged(orc, q, pool, sc), f"{what}, {n} rows, splits {splits}")
    else:
        nd, npf = int(rng.integers(0, 30)), int(rng.integers(1, 4))
        kv_d = [int(x) for x in rng.integers(1, 2000, size=nd)]
        plen = [int(x) for x in rng.integers(1, 300, size=npf)]
        prior = [int(x) for x in rng.integers(0, 500, size=npf)]
        kv = kv_d + [p + n for p, n in zip(prior, plen)]
        qlens = [1] * nd + plen
        cu = G.cu_from_lens(qlens)
        _, pool = G.decode_case(kv, hq, hkv, d, seed=case * 11 + 5)
        q = G.normal_bf16((cu[-1], hq, d), case * 11 + 9, "cuda")
        o = G.gpu_paged(q, pool, hq, hkv, d, sc, cu_q=cu, num_decode=nd, max_seqlen_q=max(qlens))
        G.assert_parity(o, G.oracle_paged(orc, q, pool, sc, cu_q=cu),
                        f"{what}, {nd} decode rows, pieces {plen} after {prior}")


@pytest.mark.parametrize("seed", [11, 23, 31])
def test_random_shapes(orc, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    for case in range(40):
        _case(orc, rng, case)
