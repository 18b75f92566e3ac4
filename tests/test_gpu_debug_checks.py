"""Debug mode (RAG_ATTN_CHECK=1): the library copies the device index arrays
(cu_seqlens, kv_lens, block tables, slot mappings) to the host before each
launch and rejects any that break a documented precondition with
RAG_ERR_INVALID_ARG, enqueueing nothing; valid arrays pass unchanged.  The
mode is read once per process, so the calls run in a child process.
"""
import json
import os
import subprocess
import sys

import pytest

from paper_2412_10543_amd import binding

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
OK, BAD = binding.RAG_OK, binding.RAG_ERR_INVALID_ARG
EXPECTED = {
    "prefill_valid": OK,
    "prefill_not_monotone": BAD,
    "prefill_over_max_seqlen": BAD,
    "prefill_more_rows_than_keys": BAD,
    "prefill_suffix_rows": OK,
    "decode_valid": OK,
    "decode_kv_len_zero": BAD,
    "decode_kv_len_past_table": BAD,
    "decode_block_id_too_large": BAD,
    "decode_block_id_negative": BAD,
    "decode_unused_entry_ignored": OK,
    "mixed_valid": OK,
    "mixed_decode_row_with_two_rows": BAD,
    "mixed_piece_longer_than_keys": BAD,
    "kv_write_valid": OK,
    "kv_write_duplicate_slot": BAD,
    "kv_write_slot_past_pool": BAD,
}


def test_debug_mode_checks_device_arrays():
    env = dict(os.environ, RAG_ATTN_CHECK="1")
    r = subprocess.run([sys.executable, "-u", os.path.join(HERE, "debug_checks_child.py")],
                       env=env, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    line = [x for x in r.stdout.splitlines() if x.startswith("{")][-1]
    got = json.loads(line)
    assert got == EXPECTED
