// Host-side configuration planner of the C ABI (declared in
// include/rag_attn.h): pruning a query profile to a configuration space
// (Algorithm 1), the KV-memory requirement of a configuration, the
// memory-aware best-fit choice with its no-fit fallback (Sec. "Joint
// configuration-scheduling adaptation"), and the device's free memory.
#include <hip/hip_runtime.h>

#include "errors.h"
#include "rag_attn.h"

namespace {

using rag::fail;

constexpr uint32_t bit(int m) { return 1u << m; }

// KV memory of `tokens` tokens with the 2% buffer, rounded up to a byte.
int64_t kv_of(int64_t tokens, int64_t bpt) { return (tokens * bpt * 102 + 99) / 100; }

// Memory a configuration needs free to start: one quantity, used both to
// decide whether it fits and to rank the configurations that do.  A call
// holds its prompt and the tokens it generates.  stuff: its one call of
// n*C + Lq prompt tokens; map_rerank: its n calls of C + Lq, which run
// together; map_reduce: its largest single call -- a mapper of C + Lq that
// writes `il` summary tokens, or the reduce call of n*il + Lq -- because the
// mappers enter the running batch one by one as memory allows and the reduce
// call starts after they have finished.
int64_t requirement_of(int method, int64_t n, int64_t il, const rag_request_shape& s) {
  const int64_t bpt = s.kv_bytes_per_token;
  const int64_t c = s.chunk_len, q = s.query_len, a = s.answer_len;
  if (method == RAG_STUFF) return kv_of(n * c + q + a, bpt);
  if (method == RAG_MAP_RERANK) return kv_of(n * (c + q + a), bpt);
  const int64_t one_mapper = kv_of(c + q + il, bpt);
  const int64_t reduce = kv_of(n * il + q + a, bpt);
  return one_mapper > reduce ? one_mapper : reduce;
}

rag_status check_shape(const rag_request_shape* s) {
  if (!s) return fail(RAG_ERR_INVALID_ARG, "planner: null request shape");
  if (s->query_len < 0 || s->chunk_len < 0 || s->answer_len < 0 || s->kv_bytes_per_token <= 0)
    return fail(RAG_ERR_INVALID_ARG, "planner: request shape needs non-negative lengths and "
                                     "positive bytes per token");
  if (s->kv_bytes_per_token > ((int64_t)1 << 32) || s->chunk_len > (1 << 24) ||
      s->query_len > (1 << 24) || s->answer_len > (1 << 24))
    return fail(RAG_ERR_INVALID_ARG, "planner: request shape out of range");
  return RAG_OK;
}

rag_status check_profile(const rag_query_profile* p) {
  if (!p) return fail(RAG_ERR_INVALID_ARG, "planner: null query profile");
  if ((p->complexity_high != 0 && p->complexity_high != 1) ||
      (p->joint_reasoning != 0 && p->joint_reasoning != 1))
    return fail(RAG_ERR_INVALID_ARG, "planner: complexity and joint reasoning are 0 or 1");
  if (p->pieces < 1 || p->pieces > (1 << 16))
    return fail(RAG_ERR_INVALID_ARG, "planner: pieces of information %d out of range", p->pieces);
  if (p->summary_len_min < 1 || p->summary_len_max < p->summary_len_min ||
      p->summary_len_max > (1 << 16))
    return fail(RAG_ERR_INVALID_ARG, "planner: bad summary length range [%d, %d]",
                p->summary_len_min, p->summary_len_max);
  return RAG_OK;
}

}  // namespace

extern "C" {

rag_status rag_prune_config_space(const rag_query_profile* profile, rag_config_space* space) {
  const rag_status st = check_profile(profile);
  if (st != RAG_OK) return st;
  if (!space) return fail(RAG_ERR_INVALID_ARG, "planner: null config space");
  // Algorithm 1: the method from joint reasoning and complexity, 1-3x the
  // pieces of information as chunks, the summary range as intermediate length.
  if (!profile->joint_reasoning)
    space->methods = bit(RAG_MAP_RERANK);
  else if (!profile->complexity_high)
    space->methods = bit(RAG_STUFF);
  else
    space->methods = bit(RAG_STUFF) | bit(RAG_MAP_REDUCE_MAP);
  space->num_chunks_min = profile->pieces;
  space->num_chunks_max = 3 * profile->pieces;
  space->intermediate_length_min = profile->summary_len_min;
  space->intermediate_length_max = profile->summary_len_max;
  return rag::ok();
}

int64_t rag_config_kv_bytes(int32_t method, int32_t num_chunks, int32_t intermediate_length,
                            const rag_request_shape* shape) {
  if (check_shape(shape) != RAG_OK || num_chunks < 0 || intermediate_length < 0) return -1;
  if (method != RAG_STUFF && method != RAG_MAP_REDUCE_MAP && method != RAG_MAP_RERANK) return -1;
  return requirement_of(method, num_chunks, intermediate_length, *shape);
}

rag_status rag_choose_config(const rag_query_profile* profile, const rag_request_shape* shape,
                             int64_t available_bytes, rag_config* out) {
  rag_status st = check_profile(profile);
  if (st != RAG_OK) return st;
  st = check_shape(shape);
  if (st != RAG_OK) return st;
  if (!out) return fail(RAG_ERR_INVALID_ARG, "planner: null output");
  if (available_bytes < 0) return fail(RAG_ERR_INVALID_ARG, "planner: negative available memory");
  rag_config_space sp;
  rag_prune_config_space(profile, &sp);
  // Best fit: the configuration of the pruned space with the highest memory
  // requirement among those whose requirement fits in the available memory;
  // ties go to more chunks, a longer intermediate length, then stuff,
  // map_reduce, map_rerank in that order.
  bool found = false;
  rag_config best{};
  const int order[3] = {RAG_STUFF, RAG_MAP_REDUCE_MAP, RAG_MAP_RERANK};
  for (int mi = 0; mi < 3; ++mi) {
    const int m = order[mi];
    if (!(sp.methods & bit(m))) continue;
    const int il_lo = m == RAG_MAP_REDUCE_MAP ? sp.intermediate_length_min : 0;
    const int il_hi = m == RAG_MAP_REDUCE_MAP ? sp.intermediate_length_max : 0;
    for (int n = sp.num_chunks_min; n <= sp.num_chunks_max; ++n)
      for (int il = il_lo; il <= il_hi; ++il) {
        const int64_t need = requirement_of(m, n, il, *shape);
        if (need > available_bytes) continue;
        const bool better =
            !found || need > best.kv_bytes ||
            (need == best.kv_bytes &&
             (n > best.num_chunks ||
              (n == best.num_chunks && il > best.intermediate_length)));
        if (better) {
          best = rag_config{m, n, il, 0, need};
          found = true;
        }
      }
  }
  if (!found) {
    // Nothing in the pruned space can start: a cheaper fixed method just
    // outside it -- stuff if joint reasoning is needed, else map_rerank --
    // with as many chunks as fit; if not even one chunk fits, the request waits.
    const int m = profile->joint_reasoning ? RAG_STUFF : RAG_MAP_RERANK;
    for (int n = sp.num_chunks_max; n >= 1 && !found; --n) {
      const int64_t need = requirement_of(m, n, 0, *shape);
      if (need <= available_bytes) {
        best = rag_config{m, n, 0, 1, need};
        found = true;
      }
    }
  }
  if (!found) {
    *out = rag_config{-1, 0, 0, 1, 0};
    rag::ok();
    return RAG_NO_FIT;
  }
  *out = best;
  return rag::ok();
}

rag_status rag_device_free_memory(size_t* free_bytes, size_t* total_bytes) {
  if (!free_bytes || !total_bytes) return fail(RAG_ERR_INVALID_ARG, "planner: null pointer");
  const hipError_t e = hipMemGetInfo(free_bytes, total_bytes);
  if (e != hipSuccess) return fail(RAG_ERR_HIP, "hipMemGetInfo: %s", hipGetErrorString(e));
  return rag::ok();
}

}  // extern "C"
