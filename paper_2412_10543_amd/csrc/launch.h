// Host-side launch descriptors for the gfx950 kernels (internal).
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <stddef.h>
#include <stdint.h>

#include "rag_attn.h"

namespace rag {

struct PrefillArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  const int32_t* cu_q;
  const int32_t* cu_k;
  int num_seqs, max_seqlen_q, hq, hkv, d, causal;
  float scale;
  // fused paged KV-cache write (prompt prefill); slots == null: none
  void* k_cache = nullptr;
  void* v_cache = nullptr;
  const int32_t* slots = nullptr;
};

struct PagedArgs {
  const void* q;
  const void* k_cache;
  const void* v_cache;
  void* o;
  const int32_t* block_tables;
  const int32_t* kv_lens;
  const int32_t* cu_q;          // null: pure decode
  int num_seqs, num_decode, max_blocks, max_seqlen_q;
  int hq, hkv, d, num_splits;
  int slots = 0;                // partial-result slots per (row, head) in the workspace
  int bal_units = 0;            // pure decode: balanced units per kv head (0: uniform splits)
  float scale;
  float* part_o;                // workspace (null when num_splits == 1)
  float* part_lse;
  int* arrivals;
  // pure decode only: the step's new tokens [num_seqs, hkv, d], appended to
  // the cache and attended by the same launch (null: none)
  const void* k_new = nullptr;
  const void* v_new = nullptr;
};

struct KvWriteArgs {
  const void* k;                // [num_tokens, hkv, d]
  const void* v;
  void* k_cache;                // [num_blocks, hkv, 16, d]
  void* v_cache;
  const int32_t* slots;         // [num_tokens]
  int64_t num_tokens;
  int hkv, d;
};

// Launch-grid sizes, exposed so the host can check them before launching.
int64_t prefill_grid(int num_seqs, int hkv, int group, int max_seqlen_q);
int64_t paged_prefill_grid(int num_pieces, int hkv, int group, int max_seqlen_q);
int64_t paged_decode_grid(int num_decode, int hkv, int num_splits);

hipError_t launch_prefill_varlen(const PrefillArgs& a, hipStream_t stream);
hipError_t launch_paged(const PagedArgs& a, hipStream_t stream);
int64_t kv_cache_write_grid(int64_t num_tokens, int hkv, int d);
hipError_t launch_kv_cache_write(const KvWriteArgs& a, hipStream_t stream);

// Static per-device scratch of rag_attn_decode_paged_noalloc
// (decode_scratch.hip): sets it up on the current device at the first call,
// checks the sizes against its fixed capacity and returns the device
// addresses of its zeroed counter region and of its partial-result region.
rag_status decode_scratch(size_t counters, size_t partial_bytes, hipStream_t stream,
                          int** counters_out, char** partials_out);
size_t decode_scratch_capacity();

}  // namespace rag
