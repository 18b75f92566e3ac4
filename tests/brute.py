"""Pure-Python brute-force attention for tiny inputs.

Independent of the oracle: it builds the visibility mask as an explicit
matrix, exponentiates raw scores (no maximum subtracted) and sums with
``math.fsum``.  It is only usable on small, well-scaled inputs.
"""
import math


def mask_matrix(nq, nk, causal):
    """mask[i][j] is True when query row i may attend to key j.  Causal
    masking is bottom-right aligned (the query rows are the last nq of the
    nk tokens)."""
    return [[(not causal) or (j <= (nk - nq) + i) for j in range(nk)]
            for i in range(nq)]


def attend(qrows, krows, vrows, scale, causal=True):
    """qrows [nq][d], krows/vrows [nk][d] (python floats).
    Returns (o [nq][d], lse [nq])."""
    nq, nk = len(qrows), len(krows)
    d = len(vrows[0]) if nk else 0
    m = mask_matrix(nq, nk, causal)
    out, lses = [], []
    for i in range(nq):
        e = [math.exp(scale * math.fsum(a * b for a, b in zip(qrows[i], krows[j])))
             if m[i][j] else 0.0 for j in range(nk)]
        z = math.fsum(e)
        out.append([math.fsum(e[j] * vrows[j][c] for j in range(nk)) / z
                    for c in range(d)])
        lses.append(math.log(z))
    return out, lses


def varlen(q, k, v, cu_q, cu_k, scale, causal=True):
    """q [Tq][hq][d], k/v [Tk][hkv][d] nested lists.  Returns (o, lse[hq][Tq])."""
    hq, hkv = len(q[0]), len(k[0])
    group = hq // hkv
    o = [[None] * hq for _ in range(len(q))]
    lse = [[None] * len(q) for _ in range(hq)]
    for s in range(len(cu_q) - 1):
        for h in range(hq):
            g = h // group
            qs = [q[r][h] for r in range(cu_q[s], cu_q[s + 1])]
            ks = [k[r][g] for r in range(cu_k[s], cu_k[s + 1])]
            vs = [v[r][g] for r in range(cu_k[s], cu_k[s + 1])]
            if not qs:
                continue
            oo, ll = attend(qs, ks, vs, scale, causal)
            for i, r in enumerate(range(cu_q[s], cu_q[s + 1])):
                o[r][h] = oo[i]
                lse[h][r] = ll[i]
    return o, lse


def paged(q, k_cache, v_cache, block_tables, kv_lens, scale, cu_q=None):
    """q [Tq][hq][d]; caches [nb][hkv][bs][d]; one query row per sequence
    when cu_q is None.  Returns (o, lse[hq][Tq])."""
    hq, hkv, bs = len(q[0]), len(k_cache[0]), len(k_cache[0][0])
    group = hq // hkv
    ns = len(kv_lens)
    cu = cu_q if cu_q is not None else list(range(ns + 1))
    o = [[None] * hq for _ in range(len(q))]
    lse = [[None] * len(q) for _ in range(hq)]
    for s in range(ns):
        for h in range(hq):
            g = h // group
            ks, vs = [], []
            for j in range(kv_lens[s]):
                blk = block_tables[s][j // bs]
                ks.append(k_cache[blk][g][j % bs])
                vs.append(v_cache[blk][g][j % bs])
            qs = [q[r][h] for r in range(cu[s], cu[s + 1])]
            oo, ll = attend(qs, ks, vs, scale, True)
            for i, r in enumerate(range(cu[s], cu[s + 1])):
                o[r][h] = oo[i]
                lse[h][r] = ll[i]
    return o, lse
