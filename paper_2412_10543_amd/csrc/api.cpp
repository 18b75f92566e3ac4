// C ABI of librag_attn (declared in include/rag_attn.h): argument
// validation, split policy, optional device-array checks, the prompt planner.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "errors.h"
#include "launch.h"
#include "rag_attn.h"

namespace {
thread_local std::string g_last_error;
}  // namespace

namespace rag {

rag_status fail(rag_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

rag_status ok() {
  g_last_error.clear();
  return RAG_OK;
}

}  // namespace rag

namespace {

using rag::fail;
using rag::ok;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool check_mode() {
  static const bool on = [] {
    const char* e = std::getenv("RAG_ATTN_CHECK");
    return e != nullptr && e[0] == '1';
  }();
  return on;
}

// Copies n int32 values from device memory (stream-ordered, synchronous).
bool fetch(std::vector<int32_t>& dst, const int32_t* src, size_t n, hipStream_t stream) {
  dst.resize(n);
  if (n == 0) return true;
  if (hipMemcpyAsync(dst.data(), src, n * sizeof(int32_t), hipMemcpyDeviceToHost, stream) !=
      hipSuccess)
    return false;
  return hipStreamSynchronize(stream) == hipSuccess;
}

rag_status check_cu(const std::vector<int32_t>& cu, const char* name, int32_t max_len) {
  if (cu[0] != 0) return fail(RAG_ERR_INVALID_ARG, "%s[0] = %d, expected 0", name, cu[0]);
  for (size_t s = 0; s + 1 < cu.size(); ++s) {
    const int64_t n = (int64_t)cu[s + 1] - cu[s];
    if (n < 0) return fail(RAG_ERR_INVALID_ARG, "%s decreases at %zu", name, s);
    if (n > max_len)
      return fail(RAG_ERR_INVALID_ARG, "%s: sequence %zu has %lld > max %d rows", name, s,
                  (long long)n, max_len);
  }
  return RAG_OK;
}

constexpr int32_t kBlock = 16;
constexpr int32_t kMaxGroupDecode = 16;
// Decode units are workgroups of four waves.  Each unit pays a fixed cost
// (first page latency, merge of its split), so auto splits aim at about one
// unit per CU, cap a unit at 512 pages (load balance across sequences of very
// different length) and keep at least 16 pages per unit (two steps per
// wave).  The in-kernel merge handles at most 64 splits.
constexpr int32_t kTargetUnits = 256;
constexpr int32_t kMaxPagesPerUnit = 512;
constexpr int32_t kMinPagesPerUnit = 16;
constexpr int32_t kMaxSplits = 64;

int32_t auto_splits(int32_t num_decode, int32_t hkv, int32_t max_blocks) {
  const int64_t base = std::max<int64_t>(1, (int64_t)num_decode * hkv);
  int64_t n = (kTargetUnits + base - 1) / base;
  n = std::max<int64_t>(n, (max_blocks + kMaxPagesPerUnit - 1) / kMaxPagesPerUnit);
  n = std::min<int64_t>(n, std::max<int64_t>(1, (max_blocks + kMinPagesPerUnit - 1) /
                                                     kMinPagesPerUnit));
  return (int32_t)std::max<int64_t>(1, n);
}

int32_t resolve_splits(int32_t num_decode, int32_t hkv, int32_t max_blocks, int32_t requested) {
  int32_t n = requested > 0 ? requested : auto_splits(num_decode, hkv, max_blocks);
  n = std::max(1, std::min({n, std::max(1, max_blocks), kMaxSplits}));
  // No split may be empty for the longest sequence: shrink to ceil(P / pps).
  const int32_t pps = (max_blocks + n - 1) / n;
  return std::max(1, (max_blocks + pps - 1) / pps);
}

// Balanced units per kv head for a pure decode launch with the automatic
// policy when its (row, kv head) pairs are fewer than the units aimed at: the
// pages of all rows are cut into equal ranges, so that rows of very different
// lengths still give every CU the same amount to stream.  0: not used.
int32_t balanced_units(int32_t num_decode, int32_t hkv, int32_t max_blocks, int32_t requested) {
  // (the kernel plans over at most 4 x 64 rows, which this bound implies)
  if (requested > 0 || num_decode <= 0 || (int64_t)num_decode * hkv >= kTargetUnits) return 0;
  // ... and no more units than pages / kMinPagesPerUnit (what the kernel uses)
  const int64_t pages = (int64_t)num_decode * std::max(max_blocks, 1);
  const int64_t units = std::min<int64_t>({kMaxSplits, (kTargetUnits + hkv - 1) / hkv,
                                           pages / kMinPagesPerUnit});
  if (units <= 1) return 0;
  // the kernel's page arithmetic is 32-bit
  if (pages * (units + 1) >= ((int64_t)1 << 31)) return 0;
  return (int32_t)units;
}

// Partial-result slots per decode row: the most pieces either policy cuts a
// row into (this sizes the workspace whichever launch uses it).
int32_t decode_slots(int32_t num_decode, int32_t hkv, int32_t max_blocks, int32_t requested) {
  return std::max(resolve_splits(num_decode, hkv, max_blocks, requested),
                  balanced_units(num_decode, hkv, max_blocks, requested));
}

// Workspace: [arrival counters int32, one per (decode row, kv head)]
// [partial outputs fp32] [partial log-sum-exp fp32], each 256-byte aligned.
struct WsLayout {
  size_t o_off, lse_off, bytes;
};

WsLayout workspace_layout(int32_t num_decode, int32_t hq, int32_t hkv, int32_t d,
                          int32_t splits) {
  WsLayout w{0, 0, 0};
  if (splits <= 1 || num_decode <= 0) return w;
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t rows = (size_t)num_decode * hq * splits;
  w.o_off = up((size_t)num_decode * hkv * sizeof(int32_t));
  w.lse_off = w.o_off + up(rows * d * sizeof(float));
  w.bytes = w.lse_off + up(rows * sizeof(float));
  return w;
}

// Debug-mode check of a slot mapping: in range, no slot written twice.
rag_status check_slots(const std::vector<int32_t>& sl, int32_t num_blocks, const char* who) {
  const int64_t slots = (int64_t)num_blocks * kBlock;
  std::vector<char> seen((size_t)std::max<int64_t>(slots, 0), 0);
  for (size_t t = 0; t < sl.size(); ++t) {
    const int32_t s = sl[t];
    if (s < 0) continue;
    if (s >= slots)
      return fail(RAG_ERR_INVALID_ARG, "%s: slot_mapping[%zu] = %d outside [0, %lld)", who, t, s,
                  (long long)slots);
    if (seen[(size_t)s]++)
      return fail(RAG_ERR_INVALID_ARG, "%s: slot %d is written by two tokens", who, s);
  }
  return RAG_OK;
}

// The prefill behind both entry points; k_cache/v_cache/slots non-null: the
// prompt prefill that also stores every K/V row in the paged cache.
rag_status prefill_impl(const void* q, const void* k, const void* v, void* o, float* lse,
                        const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k,
                        int32_t num_seqs, int32_t max_seqlen_q, int32_t max_seqlen_k,
                        int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                        float softmax_scale, int32_t causal, hipStream_t stream,
                        void* k_cache = nullptr, void* v_cache = nullptr,
                        const int32_t* slots = nullptr, int32_t num_blocks = 0) {
  if (!q || !k || !v || !o || !cu_seqlens_q || !cu_seqlens_k)
    return fail(RAG_ERR_INVALID_ARG, "prefill: null pointer argument");
  if (num_seqs < 0 || max_seqlen_q < 0 || max_seqlen_k < 0)
    return fail(RAG_ERR_INVALID_ARG, "prefill: negative size");
  if (num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads != 0)
    return fail(RAG_ERR_INVALID_ARG, "prefill: num_q_heads %d must be a positive multiple of "
                                     "num_kv_heads %d", num_q_heads, num_kv_heads);
  if (causal != 0 && causal != 1) return fail(RAG_ERR_INVALID_ARG, "prefill: causal must be 0/1");
  if (!(softmax_scale > 0.f) || softmax_scale > 1e30f)
    return fail(RAG_ERR_INVALID_ARG, "prefill: softmax_scale must be positive and finite");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return fail(RAG_ERR_INVALID_ARG, "prefill: q/k/v/o must be 16-byte aligned");
  if (head_dim != 64 && head_dim != 128)
    return fail(RAG_ERR_UNSUPPORTED, "prefill: head_dim %d (supported: 64, 128)", head_dim);
  if (num_seqs == 0 || max_seqlen_q == 0) return ok();
  const int64_t grid = rag::prefill_grid(num_seqs, num_kv_heads, num_q_heads / num_kv_heads,
                                         max_seqlen_q);
  if (grid > INT_MAX) return fail(RAG_ERR_UNSUPPORTED, "prefill: batch too large for one grid");

  if (check_mode()) {
    std::vector<int32_t> cq, ck;
    if (!fetch(cq, cu_seqlens_q, num_seqs + 1, stream) ||
        !fetch(ck, cu_seqlens_k, num_seqs + 1, stream))
      return fail(RAG_ERR_HIP, "prefill: debug copy of cu_seqlens failed");
    rag_status st = check_cu(cq, "cu_seqlens_q", max_seqlen_q);
    if (st != RAG_OK) return st;
    st = check_cu(ck, "cu_seqlens_k", max_seqlen_k);
    if (st != RAG_OK) return st;
    if (causal)
      for (int32_t s = 0; s < num_seqs; ++s)
        if (cq[s + 1] - cq[s] > ck[s + 1] - ck[s])
          return fail(RAG_ERR_INVALID_ARG, "prefill: sequence %d has more query rows than keys", s);
    if (slots) {
      std::vector<int32_t> sl;
      if (!fetch(sl, slots, (size_t)ck[num_seqs], stream))
        return fail(RAG_ERR_HIP, "prefill kvcache: debug copy of slot_mapping failed");
      rag_status st2 = check_slots(sl, num_blocks, "prefill kvcache");
      if (st2 != RAG_OK) return st2;
    }
  }

  rag::PrefillArgs a{q, k, v, o, lse, cu_seqlens_q, cu_seqlens_k, num_seqs, max_seqlen_q,
                     num_q_heads, num_kv_heads, head_dim, causal, softmax_scale};
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.slots = slots;
  const hipError_t e = rag::launch_prefill_varlen(a, stream);
  if (e != hipSuccess) return fail(RAG_ERR_HIP, "prefill launch: %s", hipGetErrorString(e));
  return ok();
}

// The decode call behind both entry points.  scratch == false: the split
// partials go to the caller's workspace (standard layout).  scratch == true:
// to the library's static per-device scratch (rag::decode_scratch); workspace
// and workspace_bytes are then unused.
rag_status decode_paged_impl(const void* q, const void* k_cache, const void* v_cache, void* o,
                             const int32_t* block_tables, const int32_t* kv_lens,
                             const int32_t* cu_seqlens_q, int32_t num_seqs,
                             int32_t num_decode_seqs, int32_t max_blocks_per_seq,
                             int32_t max_seqlen_q, int32_t num_blocks, int32_t num_q_heads,
                             int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                             float softmax_scale, int32_t num_splits, void* workspace,
                             size_t workspace_bytes, bool scratch, hipStream_t stream,
                             const void* k_new = nullptr, const void* v_new = nullptr) {
  if (!q || !k_cache || !v_cache || !o || !block_tables || !kv_lens)
    return fail(RAG_ERR_INVALID_ARG, "decode: null pointer argument");
  if (num_seqs < 0 || max_blocks_per_seq < 0 || num_blocks < 0 || max_seqlen_q < 0 ||
      num_splits < 0)
    return fail(RAG_ERR_INVALID_ARG, "decode: negative size");
  if (num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads != 0)
    return fail(RAG_ERR_INVALID_ARG, "decode: num_q_heads %d must be a positive multiple of "
                                     "num_kv_heads %d", num_q_heads, num_kv_heads);
  if (!(softmax_scale > 0.f) || softmax_scale > 1e30f)
    return fail(RAG_ERR_INVALID_ARG, "decode: softmax_scale must be positive and finite");
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(o))
    return fail(RAG_ERR_INVALID_ARG, "decode: q/k_cache/v_cache/o must be 16-byte aligned");
  if (head_dim != 64 && head_dim != 128)
    return fail(RAG_ERR_UNSUPPORTED, "decode: head_dim %d (supported: 64, 128)", head_dim);
  if (block_size != kBlock)
    return fail(RAG_ERR_UNSUPPORTED, "decode: block_size %d (supported: 16)", block_size);
  const int32_t num_decode = cu_seqlens_q ? num_decode_seqs : num_seqs;
  if (num_decode < 0 || num_decode > num_seqs)
    return fail(RAG_ERR_INVALID_ARG, "decode: num_decode_seqs %d outside [0, %d]",
                num_decode_seqs, num_seqs);
  if (num_decode > 0 && num_q_heads / num_kv_heads > kMaxGroupDecode)
    return fail(RAG_ERR_UNSUPPORTED, "decode: %d q heads per kv head (max %d)",
                num_q_heads / num_kv_heads, kMaxGroupDecode);
  if (num_seqs == 0) return ok();
  if (max_blocks_per_seq == 0) return fail(RAG_ERR_INVALID_ARG, "decode: max_blocks_per_seq is 0");

  const int32_t splits =
      num_decode > 0 ? resolve_splits(num_decode, num_kv_heads, max_blocks_per_seq, num_splits)
                     : 1;
  const int32_t slots =
      num_decode > 0 ? decode_slots(num_decode, num_kv_heads, max_blocks_per_seq, num_splits) : 1;
  const int32_t bal = cu_seqlens_q == nullptr
                          ? balanced_units(num_decode, num_kv_heads, max_blocks_per_seq, num_splits)
                          : 0;
  const WsLayout ws = workspace_layout(num_decode, num_q_heads, num_kv_heads, head_dim, slots);
  const size_t need = ws.bytes;
  if (!scratch && need > 0 && (workspace == nullptr || workspace_bytes < need))
    return fail(RAG_ERR_WORKSPACE, "decode: workspace of %zu bytes needed, %zu given", need,
                workspace == nullptr ? (size_t)0 : workspace_bytes);
  if (!scratch && need > 0 && (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
    return fail(RAG_ERR_INVALID_ARG, "decode: workspace must be 256-byte aligned");
  const int32_t group = num_q_heads / num_kv_heads;
  const bool mixed = cu_seqlens_q != nullptr && num_seqs > num_decode;
  const int64_t grid =
      (mixed ? rag::paged_prefill_grid(num_seqs - num_decode, num_kv_heads, group, max_seqlen_q)
             : 0) +
      std::max<int64_t>(rag::paged_decode_grid(num_decode, num_kv_heads, splits),
                        (int64_t)bal * num_kv_heads) + 8;   // + group padding
  if (grid > INT_MAX) return fail(RAG_ERR_UNSUPPORTED, "decode: batch too large for one grid");

  if (check_mode()) {
    std::vector<int32_t> kl, bt, cq;
    if (!fetch(kl, kv_lens, num_seqs, stream) ||
        !fetch(bt, block_tables, (size_t)num_seqs * max_blocks_per_seq, stream) ||
        (cu_seqlens_q && !fetch(cq, cu_seqlens_q, num_seqs + 1, stream)))
      return fail(RAG_ERR_HIP, "decode: debug copy of device arrays failed");
    if (cu_seqlens_q) {
      rag_status st = check_cu(cq, "cu_seqlens_q", std::max(max_seqlen_q, 1));
      if (st != RAG_OK) return st;
    }
    for (int32_t s = 0; s < num_seqs; ++s) {
      const int32_t n = kl[s];
      const int32_t nq = cu_seqlens_q ? cq[s + 1] - cq[s] : 1;
      if (n < 1 || (int64_t)n > (int64_t)max_blocks_per_seq * kBlock)
        return fail(RAG_ERR_INVALID_ARG, "decode: kv_lens[%d] = %d outside [1, %d]", s, n,
                    max_blocks_per_seq * kBlock);
      if (s < num_decode && nq != 1)
        return fail(RAG_ERR_INVALID_ARG, "decode: decode sequence %d has %d query rows", s, nq);
      if (nq > n)
        return fail(RAG_ERR_INVALID_ARG, "decode: sequence %d has %d query rows > %d keys", s,
                    nq, n);
      for (int32_t b = 0; b < (n + kBlock - 1) / kBlock; ++b) {
        const int32_t id = bt[(size_t)s * max_blocks_per_seq + b];
        if (id < 0 || id >= num_blocks)
          return fail(RAG_ERR_INVALID_ARG, "decode: block_tables[%d][%d] = %d outside [0, %d)",
                      s, b, id, num_blocks);
      }
    }
  }

  rag::PagedArgs a;
  a.q = q;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.o = o;
  a.block_tables = block_tables;
  a.kv_lens = kv_lens;
  a.cu_q = cu_seqlens_q;
  a.num_seqs = num_seqs;
  a.num_decode = num_decode;
  a.max_blocks = max_blocks_per_seq;
  a.max_seqlen_q = max_seqlen_q;
  a.hq = num_q_heads;
  a.hkv = num_kv_heads;
  a.d = head_dim;
  a.num_splits = splits;
  a.slots = slots;
  a.bal_units = bal;
  a.scale = softmax_scale;
  a.k_new = k_new;
  a.v_new = v_new;
  a.arrivals = nullptr;
  a.part_o = a.part_lse = nullptr;
  if (need > 0 && scratch) {
    // counters in the scratch's own counter region, partials after it
    const size_t counters = (size_t)num_decode * num_kv_heads;
    const size_t partials = need - ws.o_off;
    char* part = nullptr;
    const rag_status st = rag::decode_scratch(counters, partials, stream, &a.arrivals, &part);
    if (st != RAG_OK) return st;
    a.part_o = reinterpret_cast<float*>(part);
    a.part_lse = reinterpret_cast<float*>(part + (ws.lse_off - ws.o_off));
  } else if (need > 0) {
    char* wsb = static_cast<char*>(workspace);
    a.arrivals = reinterpret_cast<int*>(wsb);
    a.part_o = reinterpret_cast<float*>(wsb + ws.o_off);
    a.part_lse = reinterpret_cast<float*>(wsb + ws.lse_off);
  }
  const hipError_t e = rag::launch_paged(a, stream);
  if (e != hipSuccess) return fail(RAG_ERR_HIP, "decode launch: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

int rag_abi_version(void) { return RAG_ATTN_ABI_VERSION; }

const char* rag_last_error(void) { return g_last_error.c_str(); }

rag_status rag_attn_prefill_varlen(const void* q, const void* k, const void* v, void* o,
                                   float* lse, const int32_t* cu_seqlens_q,
                                   const int32_t* cu_seqlens_k, int32_t num_seqs,
                                   int32_t max_seqlen_q, int32_t max_seqlen_k,
                                   int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                   float softmax_scale, int32_t causal, hipStream_t stream) {
  return prefill_impl(q, k, v, o, lse, cu_seqlens_q, cu_seqlens_k, num_seqs, max_seqlen_q,
                      max_seqlen_k, num_q_heads, num_kv_heads, head_dim, softmax_scale, causal,
                      stream);
}

int32_t rag_attn_decode_num_splits(int32_t num_decode_seqs, int32_t num_kv_heads,
                                   int32_t max_blocks_per_seq, int32_t block_size,
                                   int32_t num_splits) {
  (void)block_size;
  if (num_decode_seqs <= 0 || num_kv_heads <= 0 || max_blocks_per_seq <= 0) return 1;
  return decode_slots(num_decode_seqs, num_kv_heads, max_blocks_per_seq, num_splits);
}

size_t rag_attn_decode_workspace_size(int32_t num_decode_seqs, int32_t num_q_heads,
                                      int32_t num_kv_heads, int32_t head_dim,
                                      int32_t max_blocks_per_seq, int32_t block_size,
                                      int32_t num_splits) {
  if (num_decode_seqs <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0)
    return 0;
  const int32_t n = rag_attn_decode_num_splits(num_decode_seqs, num_kv_heads,
                                               max_blocks_per_seq, block_size, num_splits);
  return workspace_layout(num_decode_seqs, num_q_heads, num_kv_heads, head_dim, n).bytes;
}

rag_status rag_attn_decode_paged(const void* q, const void* k_cache, const void* v_cache,
                                 void* o, const int32_t* block_tables, const int32_t* kv_lens,
                                 const int32_t* cu_seqlens_q, int32_t num_seqs,
                                 int32_t num_decode_seqs, int32_t max_blocks_per_seq,
                                 int32_t max_seqlen_q, int32_t num_blocks, int32_t num_q_heads,
                                 int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                                 float softmax_scale, int32_t num_splits, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  return decode_paged_impl(q, k_cache, v_cache, o, block_tables, kv_lens, cu_seqlens_q, num_seqs,
                           num_decode_seqs, max_blocks_per_seq, max_seqlen_q, num_blocks,
                           num_q_heads, num_kv_heads, head_dim, block_size, softmax_scale,
                           num_splits, workspace, workspace_bytes, false, stream);
}

rag_status rag_attn_decode_paged_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                         void* o, const int32_t* block_tables,
                                         const int32_t* kv_lens, const int32_t* cu_seqlens_q,
                                         int32_t num_seqs, int32_t num_decode_seqs,
                                         int32_t max_blocks_per_seq, int32_t max_seqlen_q,
                                         int32_t num_blocks, int32_t num_q_heads,
                                         int32_t num_kv_heads, int32_t head_dim,
                                         int32_t block_size, float softmax_scale,
                                         int32_t num_splits, hipStream_t stream) {
  return decode_paged_impl(q, k_cache, v_cache, o, block_tables, kv_lens, cu_seqlens_q, num_seqs,
                           num_decode_seqs, max_blocks_per_seq, max_seqlen_q, num_blocks,
                           num_q_heads, num_kv_heads, head_dim, block_size, softmax_scale,
                           num_splits, nullptr, 0, true, stream);
}

rag_status rag_attn_decode_paged_append(const void* q, const void* k_new, const void* v_new,
                                        void* k_cache, void* v_cache, void* o,
                                        const int32_t* block_tables, const int32_t* kv_lens,
                                        int32_t num_seqs, int32_t max_blocks_per_seq,
                                        int32_t num_blocks, int32_t num_q_heads,
                                        int32_t num_kv_heads, int32_t head_dim,
                                        int32_t block_size, float softmax_scale,
                                        int32_t num_splits, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  if (!k_new || !v_new) return fail(RAG_ERR_INVALID_ARG, "decode append: null k_new/v_new");
  if (!aligned16(k_new) || !aligned16(v_new))
    return fail(RAG_ERR_INVALID_ARG, "decode append: k_new/v_new must be 16-byte aligned");
  return decode_paged_impl(q, k_cache, v_cache, o, block_tables, kv_lens, nullptr, num_seqs,
                           num_seqs, max_blocks_per_seq, 1, num_blocks, num_q_heads,
                           num_kv_heads, head_dim, block_size, softmax_scale, num_splits,
                           workspace, workspace_bytes, false, stream, k_new, v_new);
}

rag_status rag_attn_prefill_varlen_kvcache(const void* q, const void* k, const void* v, void* o,
                                           float* lse, const int32_t* cu_seqlens,
                                           int32_t num_seqs, int32_t max_seqlen,
                                           int32_t num_q_heads, int32_t num_kv_heads,
                                           int32_t head_dim, float softmax_scale, void* k_cache,
                                           void* v_cache, const int32_t* slot_mapping,
                                           int32_t num_blocks, int32_t block_size,
                                           hipStream_t stream) {
  if (!k_cache || !v_cache || !slot_mapping)
    return fail(RAG_ERR_INVALID_ARG, "prefill kvcache: null cache or slot_mapping");
  if (!aligned16(k_cache) || !aligned16(v_cache))
    return fail(RAG_ERR_INVALID_ARG, "prefill kvcache: k_cache/v_cache must be 16-byte aligned");
  if (block_size != kBlock)
    return fail(RAG_ERR_UNSUPPORTED, "prefill kvcache: block_size %d (supported: 16)",
                block_size);
  if (num_blocks < 0) return fail(RAG_ERR_INVALID_ARG, "prefill kvcache: negative num_blocks");
  return prefill_impl(q, k, v, o, lse, cu_seqlens, cu_seqlens, num_seqs, max_seqlen, max_seqlen,
                      num_q_heads, num_kv_heads, head_dim, softmax_scale, 1, stream, k_cache,
                      v_cache, slot_mapping, num_blocks);
}

rag_status rag_kv_cache_write(const void* k, const void* v, void* k_cache, void* v_cache,
                              const int32_t* slot_mapping, int32_t num_tokens,
                              int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                              int32_t num_blocks, hipStream_t stream) {
  if (num_tokens < 0 || num_blocks < 0)
    return fail(RAG_ERR_INVALID_ARG, "kv write: negative size");
  if (num_kv_heads <= 0) return fail(RAG_ERR_INVALID_ARG, "kv write: num_kv_heads must be > 0");
  if (head_dim != 64 && head_dim != 128)
    return fail(RAG_ERR_UNSUPPORTED, "kv write: head_dim %d (supported: 64, 128)", head_dim);
  if (block_size != kBlock)
    return fail(RAG_ERR_UNSUPPORTED, "kv write: block_size %d (supported: 16)", block_size);
  if (num_tokens == 0) return ok();
  if (!k || !v || !k_cache || !v_cache || !slot_mapping)
    return fail(RAG_ERR_INVALID_ARG, "kv write: null pointer argument");
  if (!aligned16(k) || !aligned16(v) || !aligned16(k_cache) || !aligned16(v_cache))
    return fail(RAG_ERR_INVALID_ARG, "kv write: k/v/k_cache/v_cache must be 16-byte aligned");
  if (rag::kv_cache_write_grid(num_tokens, num_kv_heads, head_dim) > INT_MAX)
    return fail(RAG_ERR_UNSUPPORTED, "kv write: batch too large for one grid");
  if (check_mode()) {
    std::vector<int32_t> sl;
    if (!fetch(sl, slot_mapping, (size_t)num_tokens, stream))
      return fail(RAG_ERR_HIP, "kv write: debug copy of slot_mapping failed");
    const rag_status st = check_slots(sl, num_blocks, "kv write");
    if (st != RAG_OK) return st;
  }
  rag::KvWriteArgs a{k, v, k_cache, v_cache, slot_mapping, num_tokens, num_kv_heads, head_dim};
  const hipError_t e = rag::launch_kv_cache_write(a, stream);
  if (e != hipSuccess) return fail(RAG_ERR_HIP, "kv write launch: %s", hipGetErrorString(e));
  return ok();
}

rag_status rag_plan_prompts(rag_synthesis method, int32_t num_queries, const int32_t* query_len,
                            const int32_t* num_chunks, int32_t chunk_len,
                            int32_t intermediate_length, int32_t answer_len,
                            int32_t* cu_seqlens_out, int32_t capacity, int32_t* num_seqs_out,
                            int32_t* decode_len_out) {
  if (method < RAG_STUFF || method > RAG_MAP_RERANK)
    return fail(RAG_ERR_INVALID_ARG, "plan: unknown synthesis method %d", (int)method);
  if (num_queries < 0 || chunk_len < 0 || intermediate_length < 0 || answer_len < 0 ||
      capacity < 0)
    return fail(RAG_ERR_INVALID_ARG, "plan: negative size");
  if (!num_seqs_out || (num_queries > 0 && (!query_len || !num_chunks)))
    return fail(RAG_ERR_INVALID_ARG, "plan: null pointer argument");
  // Count calls first (validates per-query values).
  int64_t calls = 0;
  for (int32_t i = 0; i < num_queries; ++i) {
    if (query_len[i] < 0 || num_chunks[i] < 0)
      return fail(RAG_ERR_INVALID_ARG, "plan: query %d has a negative length or chunk count", i);
    const bool per_chunk = method == RAG_MAP_REDUCE_MAP || method == RAG_MAP_RERANK;
    calls += per_chunk ? num_chunks[i] : 1;
  }
  if (calls > INT32_MAX - 1) return fail(RAG_ERR_INVALID_ARG, "plan: too many calls");
  *num_seqs_out = (int32_t)calls;
  if (!cu_seqlens_out || capacity < calls + 1)
    return fail(RAG_ERR_WORKSPACE, "plan: capacity %d < %lld entries", capacity,
                (long long)calls + 1);
  int64_t total = 0;
  int32_t n = 0;
  cu_seqlens_out[0] = 0;
  auto emit = [&](int64_t len, int32_t dec) -> bool {
    total += len;
    if (total > INT32_MAX) return false;
    cu_seqlens_out[n + 1] = (int32_t)total;
    if (decode_len_out) decode_len_out[n] = dec;
    ++n;
    return true;
  };
  for (int32_t i = 0; i < num_queries; ++i) {
    const int64_t lq = query_len[i], nc = num_chunks[i];
    bool fine = true;
    switch (method) {
      case RAG_STUFF:  // all chunks then the query, one call
        fine = emit(nc * chunk_len + lq, answer_len);
        break;
      case RAG_MAP_REDUCE_MAP:  // one mapper per chunk, each writes a summary
        for (int64_t c = 0; c < nc && fine; ++c) fine = emit(chunk_len + lq, intermediate_length);
        break;
      case RAG_MAP_REDUCE_REDUCE:  // the summaries then the query, one call
        fine = emit(nc * intermediate_length + lq, answer_len);
        break;
      case RAG_MAP_RERANK:  // one answer per chunk
        for (int64_t c = 0; c < nc && fine; ++c) fine = emit(chunk_len + lq, answer_len);
        break;
    }
    if (!fine) return fail(RAG_ERR_INVALID_ARG, "plan: total prompt tokens overflow int32");
  }
  return ok();
}

}  // extern "C"
