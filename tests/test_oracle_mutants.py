"""Plant plausible mistakes in a copy of the oracle's C source and check that
the pins catch every one.  This shows the pins can tell a wrong oracle from a
right one; the shipped source is never modified."""
import os
import subprocess

import pytest

import oracle
import oracle_pins

SRC = open(oracle.attention.SOURCE).read()

# (name, original text, planted text).  Every edit keeps memory accesses in
# bounds for the pin inputs.
MUTANTS = [
    ("causal_off_by_one", "return (nk - nq) + i + 1;", "return (nk - nq) + i;"),
    ("causal_top_left", "return (nk - nq) + i + 1;", "return i + 1;"),
    ("causal_ignored", "if (!causal) return nk;", "return nk;"),
    ("scale_dropped", "s[j] = dot * scale;", "s[j] = dot;"),
    ("max_not_subtracted", "s[j] = exp(s[j] - m);", "s[j] = exp(s[j]);"),
    ("lse_without_log", "*lse = m + log(z);", "*lse = m + z;"),
    ("no_normalisation", "const double w = s[j] / z;", "const double w = s[j];"),
    ("weights_unnormalised_out", "if (p) p[j] = w;", "if (p) p[j] = s[j];"),
    ("values_from_keys", "vr[j] = v + ((size_t)(k0 + j) * hkv + g) * d;",
     "vr[j] = k + ((size_t)(k0 + j) * hkv + g) * d;"),
    ("reversed_dot", "dot += q[c] * krow[j][c];", "dot += q[c] * krow[j][d - 1 - c];"),
    ("gqa_modulo", "const int32_t g = (int32_t)(((int64_t)h * hkv) / hq);\n      const int32_t q0 = cu_q[s]",
     "const int32_t g = h % hkv;\n      const int32_t q0 = cu_q[s]"),
    ("keys_offset_from_queries", "const int32_t k0 = cu_k[s], nk = cu_k[s + 1] - cu_k[s];",
     "const int32_t k0 = cu_q[s], nk = cu_k[s + 1] - cu_k[s];"),
    ("page_blocks_rotated", "block_tables[(size_t)s * max_blocks + j / bs]",
     "block_tables[(size_t)s * max_blocks + (j / bs + 1) % ((nk + bs - 1) / bs)]"),
    ("page_slot_wrong", "* bs + (size_t)(j % bs)) * d;", "* bs + (size_t)(j / bs) % bs) * d;"),
    ("decode_row_zero", "const int32_t q0 = cu_q ? cu_q[s] : s;",
     "const int32_t q0 = cu_q ? cu_q[s] : 0;"),
    ("paged_gqa_first_head", "const int32_t g = (int32_t)(((int64_t)h * hkv) / hq);\n      const int32_t q0 = cu_q ? cu_q[s] : s;",
     "const int32_t g = 0;\n      const int32_t q0 = cu_q ? cu_q[s] : s;"),
    ("lse_layout_transposed", "double *lp = lse ? lse + (size_t)h * tq + row : NULL;\n        oracle_attend_row(q + (row * hq + h) * d, kr, vr,\n                          visible_keys(i, nq, nk, causal)",
     "double *lp = lse ? lse + row * hq + h : NULL;\n        oracle_attend_row(q + (row * hq + h) * d, kr, vr,\n                          visible_keys(i, nq, nk, causal)"),
]


def _build(tmp_path, name, src):
    c = tmp_path / f"{name}.c"
    c.write_text(src)
    so = tmp_path / f"lib{name}.so"
    oracle.build(str(c), str(so))
    return oracle.Oracle(str(so))


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    assert SRC.count(old) >= 1, f"mutation site for {name} not found"
    mutant = _build(tmp_path, name, SRC.replace(old, new, 1))
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(mutant)
        except AssertionError as e:
            caught.append((pin.__name__, str(e)[:80]))
    assert caught, f"no pin catches the planted mistake {name}"


def test_unmodified_copy_passes(tmp_path):
    clean = _build(tmp_path, "clean", SRC)
    for pin in oracle_pins.ALL_PINS:
        pin(clean)
