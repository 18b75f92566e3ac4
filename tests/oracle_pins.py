"""Pins for the fp64 oracle: checks against things other than the oracle itself.

Each ``pin_*`` function takes an ``oracle.Oracle`` and raises AssertionError
when the oracle disagrees with what the mathematics fixes.  ``test_oracle_pins``
runs them on the shipped oracle; ``test_oracle_mutants`` runs them on copies of
the oracle with planted mistakes and requires every mistake to be caught.

What pins what:
  brute force (pure Python, explicit mask, math.fsum)   every output and LSE
  closed forms: Q = 0 gives the mean of the visible V rows and LSE = ln(n);
    a one-key context gives that V row; a key scoring 60 above the rest
    gives its V row
  invariants: weights are a probability vector proportional to exp(score);
    adding one vector to every key changes nothing; sequence packing order and
    physical page order do not matter; paged decode equals the last row of a
    dense prefill; GQA equals MHA with repeated KV heads
  library: torch fp64 scaled_dot_product_attention with an explicit mask
"""
import math

import numpy as np

import brute


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _close(a, b, rtol=1e-12, atol=1e-12, what=""):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    err = np.abs(a - b)
    lim = atol + rtol * np.abs(b)
    assert np.all(err <= lim), f"{what}: max err {err.max():.3e}"


def _varlen_case(seed, lens_q, lens_k, hq, hkv, d):
    r = _rng(seed)
    cu_q = np.concatenate([[0], np.cumsum(lens_q)]).astype(np.int32)
    cu_k = np.concatenate([[0], np.cumsum(lens_k)]).astype(np.int32)
    q = r.standard_normal((cu_q[-1], hq, d))
    k = r.standard_normal((cu_k[-1], hkv, d))
    v = r.standard_normal((cu_k[-1], hkv, d))
    return q, k, v, cu_q, cu_k


def _paged_case(seed, kv_lens, nq, hq, hkv, d, bs):
    """Random paged batch: sequence s has nq[s] query rows and kv_lens[s]
    keys; its blocks are scattered through a shuffled pool."""
    r = _rng(seed)
    nblk = [(n + bs - 1) // bs for n in kv_lens]
    nb = sum(nblk) + 3
    perm = r.permutation(nb)
    mb = max(nblk)
    table = np.zeros((len(kv_lens), mb), dtype=np.int32)
    p = 0
    for s, b in enumerate(nblk):
        table[s, :b] = perm[p:p + b]
        p += b
    kc = r.standard_normal((nb, hkv, bs, d))
    vc = r.standard_normal((nb, hkv, bs, d))
    cu_q = np.concatenate([[0], np.cumsum(nq)]).astype(np.int32)
    q = r.standard_normal((cu_q[-1], hq, d))
    return q, kc, vc, table, np.array(kv_lens, dtype=np.int32), cu_q


def _gather_dense(kc, vc, table, kv_len, s):
    """Logical keys of sequence s as dense [n, hkv, d] arrays (test-side
    gather, independent of the oracle's)."""
    bs = kc.shape[2]
    rows_k, rows_v = [], []
    for j in range(kv_len):
        blk = table[s][j // bs]
        rows_k.append(kc[blk, :, j % bs, :])
        rows_v.append(vc[blk, :, j % bs, :])
    return np.stack(rows_k), np.stack(rows_v)


# ---------------------------------------------------------------------------
# brute force
# ---------------------------------------------------------------------------
def pin_brute_varlen_causal(orc):
    q, k, v, cu_q, cu_k = _varlen_case(11, [1, 5, 9, 3], [1, 5, 9, 3], 4, 2, 8)
    sc = 1 / math.sqrt(8)
    o, lse = orc.varlen(q, k, v, cu_q, cu_k, sc, causal=True)
    bo, bl = brute.varlen(q.tolist(), k.tolist(), v.tolist(), list(cu_q),
                          list(cu_k), sc, True)
    _close(o, bo, what="varlen causal o")
    _close(lse, bl, what="varlen causal lse")


def pin_brute_varlen_noncausal(orc):
    q, k, v, cu_q, cu_k = _varlen_case(12, [4, 7], [4, 7], 2, 1, 8)
    sc = 0.37
    o, lse = orc.varlen(q, k, v, cu_q, cu_k, sc, causal=False)
    bo, bl = brute.varlen(q.tolist(), k.tolist(), v.tolist(), list(cu_q),
                          list(cu_k), sc, False)
    _close(o, bo, what="varlen non-causal o")
    _close(lse, bl, what="varlen non-causal lse")


def pin_brute_varlen_suffix(orc):
    """Fewer query rows than keys: the query rows are the sequence's last
    tokens (chunked prefill), masked bottom-right."""
    q, k, v, cu_q, cu_k = _varlen_case(13, [1, 3, 4], [1, 6, 11], 4, 4, 8)
    sc = 1 / math.sqrt(8)
    o, lse = orc.varlen(q, k, v, cu_q, cu_k, sc, causal=True)
    bo, bl = brute.varlen(q.tolist(), k.tolist(), v.tolist(), list(cu_q),
                          list(cu_k), sc, True)
    _close(o, bo, what="suffix o")
    _close(lse, bl, what="suffix lse")


def pin_brute_paged_mixed(orc):
    """Paged batch mixing one-row decodes and multi-row chunked prefills."""
    q, kc, vc, table, kvl, cu_q = _paged_case(14, [1, 7, 16, 17, 33], [1, 1, 3, 1, 5],
                                              4, 2, 8, 4)
    sc = 1 / math.sqrt(8)
    o, lse = orc.paged(q, kc, vc, table, kvl, sc, cu_q=cu_q)
    bo, bl = brute.paged(q.tolist(), kc.tolist(), vc.tolist(), table.tolist(),
                         list(kvl), sc, cu_q=list(cu_q))
    _close(o, bo, what="paged o")
    _close(lse, bl, what="paged lse")


def pin_brute_paged_decode(orc):
    q, kc, vc, table, kvl, _ = _paged_case(15, [3, 16, 40], [1, 1, 1], 8, 2, 8, 16)
    sc = 1 / math.sqrt(8)
    o, lse = orc.paged(q, kc, vc, table, kvl, sc, cu_q=None)
    bo, bl = brute.paged(q.tolist(), kc.tolist(), vc.tolist(), table.tolist(),
                         list(kvl), sc, cu_q=None)
    _close(o, bo, what="decode o")
    _close(lse, bl, what="decode lse")


def pin_seq_rows_match_brute(orc):
    q, k, v, cu_q, cu_k = _varlen_case(16, [9], [9], 4, 2, 8)
    sc = 1 / math.sqrt(8)
    rows = np.array([0, 4, 8, 8, 2], dtype=np.int32)
    heads = np.array([0, 1, 2, 3, 3], dtype=np.int32)
    o, lse = orc.seq_rows(q[rows, heads], k, v, 9, rows, heads, 4, sc)
    bo, bl = brute.varlen(q.tolist(), k.tolist(), v.tolist(), list(cu_q),
                          list(cu_k), sc, True)
    for n, (r, h) in enumerate(zip(rows, heads)):
        _close(o[n], bo[r][h], what="seq_rows o")
        _close(lse[n], bl[h][r], what="seq_rows lse")


# ---------------------------------------------------------------------------
# closed forms
# ---------------------------------------------------------------------------
def pin_zero_query_prefix_mean(orc):
    """Q = 0 makes every visible score 0: the output is the mean of the
    visible V rows and the LSE is ln(number visible)."""
    q, k, v, cu_q, cu_k = _varlen_case(21, [6, 10], [6, 10], 2, 2, 8)
    q[:] = 0
    o, lse = orc.varlen(q, k, v, cu_q, cu_k, 0.5, causal=True)
    for s in range(2):
        for i in range(cu_q[s + 1] - cu_q[s]):
            row = cu_q[s] + i
            for h in range(2):
                want = np.mean(v[cu_k[s]:cu_k[s] + i + 1, h], axis=0)
                _close(o[row, h], want, what="prefix mean")
                _close(lse[h, row], math.log(i + 1), what="ln n")


def pin_length_one_context(orc):
    """Row 0 of a causal prefill sees one key: the output is that V row."""
    q, k, v, cu_q, cu_k = _varlen_case(22, [5, 3], [5, 3], 4, 2, 8)
    o, _ = orc.varlen(q, k, v, cu_q, cu_k, 0.3, causal=True)
    for s in range(2):
        for h in range(4):
            assert np.array_equal(o[cu_q[s], h], v[cu_k[s], h // 2]), "first row"
    q2, kc, vc, table, kvl, _ = _paged_case(23, [1, 1], [1, 1], 2, 2, 8, 16)
    o2, lse2 = orc.paged(q2, kc, vc, table, kvl, 0.3)
    for s in range(2):
        for h in range(2):
            assert np.array_equal(o2[s, h], vc[table[s, 0], h, 0]), "kv_len 1"
            _close(lse2[h, s], 0.3 * float(q2[s, h] @ kc[table[s, 0], h, 0]),
                   what="lse of one key")


def pin_dominant_key(orc):
    """One key scores 60 above every other: the output is its V row to
    within e^-60 of the others' weight."""
    r = _rng(24)
    d, n = 8, 12
    q = np.zeros((n, 1, d))
    k = r.standard_normal((n, 1, d)) * 0.01
    v = r.standard_normal((n, 1, d))
    q[n - 1, 0, 0] = 1.0
    k[5, 0, 0] = 70.0
    cu = np.array([0, n], dtype=np.int32)
    o, _ = orc.varlen(q, k, v, cu, cu, 1.0, causal=True)
    _close(o[n - 1, 0], v[5, 0], rtol=1e-20, atol=1e-20 + 1e-24 * n, what="dominant")


# ---------------------------------------------------------------------------
# invariants
# ---------------------------------------------------------------------------
def pin_weights_are_softmax(orc):
    """The weights are non-negative, sum to 1 and satisfy
    p_a / p_b = exp(s_a - s_b) for the scaled scores s."""
    r = _rng(31)
    d, n, sc = 16, 23, 0.25
    q = r.standard_normal(d)
    k = r.standard_normal((n, d)) * 2
    v = r.standard_normal((n, d))
    o, lse, p = orc.attend_row(q, k, v, sc)
    assert np.all(p >= 0)
    _close(math.fsum(p), 1.0, rtol=0, atol=1e-14, what="sum p")
    s = [sc * math.fsum(a * b for a, b in zip(q, k[j])) for j in range(n)]
    for a, b in [(0, 1), (3, 17), (22, 5), (9, 9)]:
        _close(p[a] / p[b], math.exp(s[a] - s[b]), what="ratio")
    _close(p, [math.exp(x - lse) for x in s], what="p = exp(s - lse)")
    _close(o, p @ v, what="o = p v")


def pin_key_shift_invariance(orc):
    """Adding one vector w to every key adds q.w to each score of a row,
    which the softmax removes."""
    q, k, v, cu_q, cu_k = _varlen_case(32, [7, 4], [7, 4], 2, 1, 8)
    w = _rng(33).standard_normal(8)
    o1, _ = orc.varlen(q, k, v, cu_q, cu_k, 0.4)
    o2, _ = orc.varlen(q, k + w, v, cu_q, cu_k, 0.4)
    _close(o2, o1, rtol=1e-11, atol=1e-11, what="key shift")


def pin_packing_order(orc):
    """Reordering the sequences of a packed batch reorders the outputs and
    changes nothing else (bitwise)."""
    lens = [3, 8, 1, 6]
    q, k, v, cu, _ = _varlen_case(34, lens, lens, 4, 2, 8)
    o, lse = orc.varlen(q, k, v, cu, cu, 0.35)
    order = [2, 0, 3, 1]
    segs = [(cu[s], cu[s + 1]) for s in order]
    idx = np.concatenate([np.arange(a, b) for a, b in segs])
    cu2 = np.concatenate([[0], np.cumsum([lens[s] for s in order])]).astype(np.int32)
    o2, lse2 = orc.varlen(q[idx], k[idx], v[idx], cu2, cu2, 0.35)
    assert np.array_equal(o2, o[idx]), "packing order o"
    assert np.array_equal(lse2, lse[:, idx]), "packing order lse"


def pin_page_permutation(orc):
    """Moving the pages of a sequence to other physical blocks (and updating
    the block table) changes nothing (bitwise)."""
    q, kc, vc, table, kvl, cu = _paged_case(35, [9, 30, 17], [1, 4, 2], 4, 2, 8, 4)
    o, lse = orc.paged(q, kc, vc, table, kvl, 0.3, cu_q=cu)
    perm = _rng(36).permutation(kc.shape[0])
    inv = np.argsort(perm)
    kc2 = kc[inv]
    vc2 = vc[inv]
    table2 = perm[table].astype(np.int32)
    o2, lse2 = orc.paged(q, kc2, vc2, table2, kvl, 0.3, cu_q=cu)
    assert np.array_equal(o2, o) and np.array_equal(lse2, lse), "page permutation"


def pin_decode_equals_prefill_last_row(orc):
    """A one-row decode with kv_len = L equals the last row of a causal
    prefill over the same L tokens (bitwise: same row arithmetic)."""
    q, kc, vc, table, kvl, _ = _paged_case(37, [21, 5], [1, 1], 4, 2, 8, 16)
    o, lse = orc.paged(q, kc, vc, table, kvl, 0.3)
    for s in range(2):
        kd, vd = _gather_dense(kc, vc, table, kvl[s], s)
        L = kvl[s]
        qd = np.zeros((L, 4, 8))
        qd[L - 1] = q[s]
        cu = np.array([0, L], dtype=np.int32)
        od, ld = orc.varlen(qd, kd, vd, cu, cu, 0.3)
        assert np.array_equal(od[L - 1], o[s]), "decode vs prefill o"
        assert np.array_equal(ld[:, L - 1], lse[:, s]), "decode vs prefill lse"


def pin_gqa_equals_repeated_mha(orc):
    """GQA with group size G equals MHA whose KV heads are each repeated G
    times (bitwise)."""
    q, k, v, cu, _ = _varlen_case(38, [5, 9], [5, 9], 8, 2, 8)
    o, lse = orc.varlen(q, k, v, cu, cu, 0.3)
    k4 = np.repeat(k, 4, axis=1)
    v4 = np.repeat(v, 4, axis=1)
    o2, lse2 = orc.varlen(q, k4, v4, cu, cu, 0.3)
    assert np.array_equal(o, o2) and np.array_equal(lse, lse2), "gqa vs mha"


def pin_torch_sdpa(orc):
    """torch's fp64 CPU scaled_dot_product_attention with an explicit boolean
    mask (bottom-right causal), one sequence at a time."""
    import torch
    lens_q, lens_k = [4, 9, 2], [4, 12, 7]
    q, k, v, cu_q, cu_k = _varlen_case(39, lens_q, lens_k, 4, 2, 16)
    sc = 1 / 4.0
    o, _ = orc.varlen(q, k, v, cu_q, cu_k, sc, causal=True)
    for s in range(3):
        nq, nk = lens_q[s], lens_k[s]
        qt = torch.from_numpy(q[cu_q[s]:cu_q[s + 1]]).permute(1, 0, 2)
        kt = torch.from_numpy(np.repeat(k[cu_k[s]:cu_k[s + 1]], 2, axis=1)).permute(1, 0, 2)
        vt = torch.from_numpy(np.repeat(v[cu_k[s]:cu_k[s + 1]], 2, axis=1)).permute(1, 0, 2)
        mask = torch.tensor(brute.mask_matrix(nq, nk, True))
        ref = torch.nn.functional.scaled_dot_product_attention(
            qt, kt, vt, attn_mask=mask, scale=sc).permute(1, 0, 2).numpy()
        _close(o[cu_q[s]:cu_q[s + 1]], ref, rtol=1e-10, atol=1e-12, what="sdpa")


def pin_bf16_widening(orc):
    """bf16 inputs are widened exactly: 1.0 is 0x3F80, -2.5 is 0xC020, the
    smallest bf16 subnormal is 2^-133."""
    from oracle import bf16_bits_to_f64
    bits = np.array([0x3F80, 0xC020, 0x0001, 0x7F7F], dtype=np.uint16)
    want = [1.0, -2.5, 2.0 ** -133, (2 - 2 ** -7) * 2.0 ** 127]
    assert list(bf16_bits_to_f64(bits)) == want


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
