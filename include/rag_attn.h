/*
 * rag_attn.h -- C ABI of the MI355X (gfx950) attention library for the LLM
 * synthesis step of a configuration-adaptive RAG system (METIS, arXiv
 * 2412.10543).
 *
 * Why attention: synthesis dominates a RAG query's delay (retrieval is over
 * 100x cheaper, Sec. "RAG systems and configurations"), and the three knobs the
 * system adapts per query -- num_chunks, synthesis_method (stuff, map_reduce,
 * map_rerank) and intermediate_length -- decide how many tokens that step
 * prefills and decodes.  The served models (Sec. "Setup": a 7B model with 32
 * query / 8 KV heads of size 128, a 70B model with 64 / 8) run on a serving
 * engine with a paged KV cache, continuous batching and chunked prefill (Sec.
 * "Joint configuration-scheduling adaptation", Sec. "Implementation").
 *
 * Conventions for every call:
 *   - Tensors are bf16 unless noted and row-major; "device" pointers are HIP
 *     device memory, "host" pointers host memory.  Every bf16 tensor pointer
 *     must be 16-byte aligned.
 *   - The caller owns every buffer, including workspaces.  The library never
 *     allocates or frees device memory and keeps no pointer after a call
 *     returns, apart from the work it has enqueued.
 *   - Calls enqueue on `stream` (NULL = the null stream) and return; they
 *     never synchronise (except in the debug mode below).
 *   - Host-visible arguments are validated before anything is enqueued; a
 *     failing call enqueues nothing and returns a negative rag_status.
 *     rag_last_error() then gives a message (thread-local).  No C++ exception
 *     crosses this boundary.
 *   - The contents of device arrays (cu_seqlens, kv_lens, block tables) are
 *     caller preconditions, checked only when the environment variable
 *     RAG_ATTN_CHECK=1 is set (the call then copies them to the host
 *     synchronously and returns RAG_ERR_INVALID_ARG on a violation).
 *   - Calls are thread-safe; the only mutable global state is the
 *     thread-local error message (and the static scratch of
 *     rag_attn_decode_paged_noalloc, see there).
 *   - RAG_ATTN_PF_ITEMS=n (read at each rag_attn_prefill_varlen call) fixes
 *     how many query tiles one prefill workgroup runs in sequence instead of
 *     the library's load-balancing choice; a testing and tuning knob that
 *     changes no output bit.
 *
 * Attention here is softmax(q k^T * softmax_scale) v per query row, with
 * grouped-query heads (q head h reads kv head h / (num_q_heads / num_kv_heads))
 * and causal masking aligned bottom-right: a sequence with nq query rows and
 * nk keys lets query row i (0-based) see keys j <= (nk - nq) + i.  Inputs are
 * bf16, products and softmax run in fp32, outputs are bf16 (rounded to
 * nearest even).
 */
#ifndef RAG_ATTN_H
#define RAG_ATTN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RAG_ATTN_ABI_VERSION 1

typedef enum {
  RAG_NO_FIT = 1,           /* rag_choose_config: no configuration fits in the
                               available memory; the request waits            */
  RAG_OK = 0,
  RAG_ERR_INVALID_ARG = -1, /* null pointer, negative size, bad enum, bad alignment,
                               violated precondition (debug mode)              */
  RAG_ERR_UNSUPPORTED = -2, /* valid but not implemented: head_dim not 64/128,
                               block_size not 16, GQA group over 16 in decode  */
  RAG_ERR_WORKSPACE = -3,   /* workspace missing or smaller than required     */
  RAG_ERR_HIP = -4          /* a HIP call failed (launch error, debug copy)   */
} rag_status;

/* RAG_ATTN_ABI_VERSION of the loaded library. */
int rag_abi_version(void);

/* Message for the last non-OK status returned on the calling thread ("" if
 * none).  The pointer stays valid until the next call on that thread. */
const char *rag_last_error(void);

/*
 * Packed variable-length attention: the prefill of a batch of prompts
 * assembled by rag_plan_prompts (one per stuff query, one per map_reduce
 * mapper or map_rerank chunk, one per reduce call).
 *
 *   q      device [Tq, num_q_heads, head_dim]   Tq = cu_seqlens_q[num_seqs]
 *   k, v   device [Tk, num_kv_heads, head_dim]  Tk = cu_seqlens_k[num_seqs]
 *   o      device [Tq, num_q_heads, head_dim]   output, written in full
 *   lse    device fp32 [num_q_heads, Tq] or NULL: natural-log sum of exp of
 *          the scaled scores of each row (-inf for a row that sees no key)
 *   cu_seqlens_q, cu_seqlens_k  device int32 [num_seqs + 1], non-decreasing,
 *          starting at 0.  Sequence s owns q rows [cu_q[s], cu_q[s+1]) and
 *          k/v rows [cu_k[s], cu_k[s+1]).  Precondition: with causal=1 each
 *          sequence has nq <= nk (equal for a plain prefill).
 *   max_seqlen_q  host upper bound of any nq (sizes the grid); max_seqlen_k
 *          host upper bound of any nk.
 *   causal 1: bottom-right causal mask; 0: every row sees all nk keys.
 *
 * Returns RAG_OK, RAG_ERR_INVALID_ARG (null q/k/v/o/cu pointer, num_seqs < 0,
 * heads <= 0, num_q_heads % num_kv_heads != 0, causal not 0/1, misaligned
 * pointer, max_seqlen < 0), RAG_ERR_UNSUPPORTED (head_dim not 64 or 128) or
 * RAG_ERR_HIP.  num_seqs == 0 or max_seqlen_q == 0 is a no-op.
 */
rag_status rag_attn_prefill_varlen(const void *q, const void *k, const void *v,
                                   void *o, float *lse,
                                   const int32_t *cu_seqlens_q,
                                   const int32_t *cu_seqlens_k,
                                   int32_t num_seqs, int32_t max_seqlen_q,
                                   int32_t max_seqlen_k, int32_t num_q_heads,
                                   int32_t num_kv_heads, int32_t head_dim,
                                   float softmax_scale, int32_t causal,
                                   hipStream_t stream);

/*
 * The prompt prefill with the paged KV-cache write fused in: the causal
 * attention of rag_attn_prefill_varlen over self-attention prompts (query rows
 * are the key rows: one cu_seqlens), which also stores every K and V row in
 * the paged cache rag_attn_decode_paged reads -- the step on either side of
 * the hot path in the serving engine the paper builds on (Sec.
 * "Implementation": a paged KV cache), so that decode starts on the pages with
 * no separate copy.  Each prefill workgroup writes the key rows of its own
 * query tiles after computing them, while they are still in the GPU's caches.
 *
 *   q, k, v, o, lse  as in rag_attn_prefill_varlen, with cu_seqlens_q =
 *            cu_seqlens_k = cu_seqlens and causal = 1.
 *   k_cache, v_cache  device [num_blocks, num_kv_heads, block_size, head_dim]
 *   slot_mapping  device int32 [cu_seqlens[num_seqs]]: the slot (page * 16 +
 *            offset) of each packed token; negative = not written.
 *            Precondition: slots below num_blocks * 16, none repeated (checked
 *            when RAG_ATTN_CHECK=1).  The result in the cache is that of
 *            rag_kv_cache_write(k, v, ...) with the same slot mapping.
 *   block_size  must be 16.
 *
 * Returns the statuses of rag_attn_prefill_varlen, and RAG_ERR_INVALID_ARG for
 * a null or misaligned cache or slot pointer, RAG_ERR_UNSUPPORTED for a block
 * size other than 16.
 */
rag_status rag_attn_prefill_varlen_kvcache(
    const void *q, const void *k, const void *v, void *o, float *lse,
    const int32_t *cu_seqlens, int32_t num_seqs, int32_t max_seqlen,
    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
    float softmax_scale, void *k_cache, void *v_cache,
    const int32_t *slot_mapping, int32_t num_blocks, int32_t block_size,
    hipStream_t stream);

/*
 * Partial-result slots per decode row that rag_attn_decode_paged may use when
 * it is passed num_splits (0 = choose automatically), given the number of
 * decode rows, kv heads and the block-table width: the most pieces a row's
 * keys are cut into (the workspace holds one partial output per slot).
 * Always >= 1.
 */
int32_t rag_attn_decode_num_splits(int32_t num_decode_seqs,
                                   int32_t num_kv_heads,
                                   int32_t max_blocks_per_seq,
                                   int32_t block_size, int32_t num_splits);

/*
 * Bytes of workspace rag_attn_decode_paged needs for the same arguments (0
 * when the decode rows use a single split).  Layout (library-internal): int32
 * arrival counters [num_decode_seqs, num_kv_heads], fp32 partial outputs
 * [num_decode_seqs, num_q_heads, splits, head_dim] and fp32 partial
 * log-sum-exp values [num_decode_seqs, num_q_heads, splits].
 */
size_t rag_attn_decode_workspace_size(int32_t num_decode_seqs,
                                      int32_t num_q_heads, int32_t num_kv_heads,
                                      int32_t head_dim,
                                      int32_t max_blocks_per_seq,
                                      int32_t block_size, int32_t num_splits);

/*
 * Attention of query rows against a paged KV cache: one decode step of a
 * batch, optionally mixed in the same launch with chunked-prefill pieces (the
 * engine's continuous batching with chunked prefill).
 *
 *   q        device [Tq, num_q_heads, head_dim]
 *   k_cache, v_cache  device [num_blocks, num_kv_heads, block_size, head_dim]
 *   o        device [Tq, num_q_heads, head_dim]; output
 *   block_tables  device int32 [num_seqs, max_blocks_per_seq]; entry b of row
 *            s is the physical block holding keys [16b, 16b+16) of sequence
 *            s.  Entries past ceil(kv_lens[s]/16) are never read.
 *   kv_lens  device int32 [num_seqs]: keys of sequence s, counting those of
 *            its own query rows (1 <= kv_len <= max_blocks_per_seq*16).
 *   cu_seqlens_q  device int32 [num_seqs + 1] or NULL.
 *            NULL: pure decode; sequence s has the single query row s
 *            (Tq = num_seqs) and num_decode_seqs is ignored.
 *            Non-NULL: mixed batch.  Sequences [0, num_decode_seqs) are decode
 *            rows (cu[s+1] - cu[s] == 1); sequences [num_decode_seqs,
 *            num_seqs) are chunked-prefill pieces whose nq = cu[s+1] - cu[s]
 *            query rows (0 <= nq <= max_seqlen_q, nq <= kv_len) are the last
 *            nq of their kv_len tokens.
 *   num_blocks  physical blocks in the pool (bounds for debug checks).
 *   block_size  must be 16.  head_dim 64 or 128.  The decode rows need
 *            num_q_heads / num_kv_heads <= 16.
 *   num_splits  0 = automatic; else the number of KV splits per decode row
 *            (clamped to [1, min(64, max_blocks_per_seq)]).
 *            Automatic: about one unit of work per CU.  A pure decode batch
 *            (cu_seqlens_q == NULL) with fewer (row, kv head) pairs than that
 *            has the pages of all its rows, per kv head, cut into equal
 *            ranges of at least 16 pages, so that rows of different lengths
 *            still give every unit the same amount to read; otherwise every
 *            row is cut into the same number of splits.
 *            Pieces of a row are merged (log-sum-exp) inside the same kernel
 *            by the last one to finish.
 *   workspace, workspace_bytes  device scratch of at least
 *            rag_attn_decode_workspace_size(...) bytes (may be NULL when that
 *            is 0); 256-byte aligned.  It must be zero-filled before its first
 *            use; every completed call leaves it zero-filled again (the split
 *            merge counts arrivals in it), so one zeroed buffer serves any
 *            sequence of calls.  Overlapping calls must not share it.
 *
 * Every element of o for the Tq rows is written.  Returns RAG_OK,
 * RAG_ERR_INVALID_ARG, RAG_ERR_UNSUPPORTED, RAG_ERR_WORKSPACE or RAG_ERR_HIP.
 */
rag_status rag_attn_decode_paged(const void *q, const void *k_cache,
                                 const void *v_cache, void *o,
                                 const int32_t *block_tables,
                                 const int32_t *kv_lens,
                                 const int32_t *cu_seqlens_q, int32_t num_seqs,
                                 int32_t num_decode_seqs,
                                 int32_t max_blocks_per_seq,
                                 int32_t max_seqlen_q, int32_t num_blocks,
                                 int32_t num_q_heads, int32_t num_kv_heads,
                                 int32_t head_dim, int32_t block_size,
                                 float softmax_scale, int32_t num_splits,
                                 void *workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/*
 * One decode step with the step's new token appended in the same launch: for
 * each decode row s, key kv_lens[s] - 1 is the new token, whose K and V rows
 * k_new[s], v_new[s] are stored into its cache slot (block_tables[s][(kv_lens[s]
 * - 1) / 16] * 16 + (kv_lens[s] - 1) % 16) and attended together with the keys
 * already in the cache.  Equivalent to rag_kv_cache_write of the new tokens
 * followed by rag_attn_decode_paged, in one launch (the serving engine's
 * decode iteration, Sec. "Implementation").
 *
 *   q        device [num_seqs, num_q_heads, head_dim]: one decode row per
 *            sequence (no chunked-prefill pieces)
 *   k_new, v_new  device [num_seqs, num_kv_heads, head_dim], 16-byte aligned
 *   the rest as in rag_attn_decode_paged (cu_seqlens_q = NULL).  The caches
 *            are written (one slot per sequence and kv head).
 *
 * Returns the statuses of rag_attn_decode_paged, and RAG_ERR_INVALID_ARG for a
 * null or misaligned k_new / v_new.
 */
rag_status rag_attn_decode_paged_append(
    const void *q, const void *k_new, const void *v_new, void *k_cache,
    void *v_cache, void *o, const int32_t *block_tables,
    const int32_t *kv_lens, int32_t num_seqs, int32_t max_blocks_per_seq,
    int32_t num_blocks, int32_t num_q_heads, int32_t num_kv_heads,
    int32_t head_dim, int32_t block_size, float softmax_scale,
    int32_t num_splits, void *workspace, size_t workspace_bytes,
    hipStream_t stream);

/*
 * rag_attn_decode_paged without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Arguments, results and errors are those of
 * rag_attn_decode_paged (same kernels, same split policy, bit-identical
 * outputs); the split partials and arrival counters live instead in a static
 * per-device scratch array inside the library (32 MiB per GPU the library
 * runs on, held until the process ends; set up on the current device at the
 * first call, which zeroes its counters with a small kernel on `stream`).  The
 * call allocates and frees nothing.  It returns RAG_ERR_WORKSPACE when the
 * decode rows need more than 65,536 (row, kv head) counters or more than
 * 32 MiB - 256 KiB of partials (num_decode_seqs * num_q_heads * splits *
 * (head_dim + 1) * 4 bytes, each part rounded up to 256).  Every call on a GPU
 * shares that GPU's scratch: calls that may overlap on one GPU (different
 * streams, or graphs replayed concurrently) race and must be serialised by the
 * caller.
 */
rag_status rag_attn_decode_paged_noalloc(const void *q, const void *k_cache,
                                         const void *v_cache, void *o,
                                         const int32_t *block_tables,
                                         const int32_t *kv_lens,
                                         const int32_t *cu_seqlens_q,
                                         int32_t num_seqs, int32_t num_decode_seqs,
                                         int32_t max_blocks_per_seq,
                                         int32_t max_seqlen_q, int32_t num_blocks,
                                         int32_t num_q_heads, int32_t num_kv_heads,
                                         int32_t head_dim, int32_t block_size,
                                         float softmax_scale, int32_t num_splits,
                                         hipStream_t stream);

/*
 * Paged KV-cache write: store the keys and values of a batch of new tokens in
 * the paged cache that rag_attn_decode_paged reads.  The serving engine the
 * paper builds on (Sec. "Implementation": vLLM, with its paged KV cache) keeps
 * each token's K/V in 16-token pages; a token's slot is page * 16 + offset.
 * A prefill writes its prompt tokens this way, so that decode can start on
 * the pages with no host-side re-layout; each decode step writes one token
 * per sequence.
 *
 *   k, v     device [num_tokens, num_kv_heads, head_dim]: the new tokens
 *            (for a prefill, the packed K and V given to
 *            rag_attn_prefill_varlen).
 *   k_cache, v_cache  device [num_blocks, num_kv_heads, block_size,
 *            head_dim]: token t's row of kv head h is written to
 *            cache[slot / 16][h][slot % 16][:]; nothing else changes.
 *   slot_mapping  device int32 [num_tokens]: slot of each token; a negative
 *            slot skips the token (padding).  Precondition: slots are below
 *            num_blocks * block_size and no two tokens share a slot (both
 *            checked when RAG_ATTN_CHECK=1).
 *   block_size  must be 16; head_dim 64 or 128.
 *
 * Returns RAG_OK (num_tokens == 0 is a no-op), RAG_ERR_INVALID_ARG (null or
 * misaligned pointer, negative size, num_kv_heads <= 0, violated precondition
 * in debug mode), RAG_ERR_UNSUPPORTED (head_dim, block_size) or RAG_ERR_HIP.
 */
rag_status rag_kv_cache_write(const void *k, const void *v, void *k_cache,
                              void *v_cache, const int32_t *slot_mapping,
                              int32_t num_tokens, int32_t num_kv_heads,
                              int32_t head_dim, int32_t block_size,
                              int32_t num_blocks, hipStream_t stream);

/* Synthesis methods (Sec. "RAG systems and configurations"). */
typedef enum {
  RAG_STUFF = 0,             /* one prompt: all chunks, then the query       */
  RAG_MAP_REDUCE_MAP = 1,    /* one prompt per chunk: chunk + query; each
                                decodes intermediate_length summary tokens   */
  RAG_MAP_REDUCE_REDUCE = 2, /* one prompt: the summaries, then the query    */
  RAG_MAP_RERANK = 3         /* one prompt per chunk: chunk + query; each
                                decodes an answer                            */
} rag_synthesis;

/*
 * Host-only prompt planner: the packed-batch descriptor of the LLM calls a
 * synthesis method issues for a list of queries.
 *
 *   query_len, num_chunks  host int32 [num_queries]: tokens of each query and
 *            chunks retrieved for it.
 *   chunk_len  tokens per chunk; intermediate_length  summary tokens per
 *            mapper; answer_len  tokens decoded by answer-producing calls.
 *   cu_seqlens_out  host int32 [capacity]: receives num_calls + 1 prefix
 *            offsets of the prompt lengths.
 *   num_seqs_out  host: number of calls.
 *   decode_len_out  host int32 [capacity - 1] or NULL: tokens each call
 *            decodes.
 * Prompt lengths: stuff n*chunk_len + query_len; map_reduce map and
 * map_rerank chunk_len + query_len per chunk; map_reduce reduce
 * n*intermediate_length + query_len.
 * Returns RAG_ERR_INVALID_ARG for a bad method, a null array, negative sizes
 * or a 32-bit overflow of the total, RAG_ERR_WORKSPACE when capacity is too
 * small (num_seqs_out still receives the number of calls).
 */
rag_status rag_plan_prompts(rag_synthesis method, int32_t num_queries,
                            const int32_t *query_len, const int32_t *num_chunks,
                            int32_t chunk_len, int32_t intermediate_length,
                            int32_t answer_len, int32_t *cu_seqlens_out,
                            int32_t capacity, int32_t *num_seqs_out,
                            int32_t *decode_len_out);

/*
 * Configuration planner (host only).  A query's profile -- estimated by an LLM
 * in the paper, given here -- is pruned to a space of configurations
 * (Algorithm 1, Sec. "Mapping query profiles to RAG configurations"); one
 * configuration of that space is then chosen from the GPU memory available
 * for the current batch (Sec. "Joint configuration-scheduling adaptation").
 */
typedef struct {
  int32_t complexity_high;   /* query complexity: 1 = "High", 0 = "Low"          */
  int32_t joint_reasoning;   /* joint reasoning required: 1 = "Yes", 0 = "No"    */
  int32_t pieces;            /* pieces of information required (paper: 1-10)    */
  int32_t summary_len_min;   /* length range of the summaries, tokens           */
  int32_t summary_len_max;   /*   (paper: 30-200)                               */
} rag_query_profile;

typedef struct {
  uint32_t methods;          /* bit (1u << m) for each allowed method m: RAG_STUFF,
                                RAG_MAP_REDUCE_MAP (a map_reduce configuration)
                                or RAG_MAP_RERANK                               */
  int32_t num_chunks_min, num_chunks_max;
  int32_t intermediate_length_min, intermediate_length_max;
} rag_config_space;

typedef struct {
  int32_t query_len;         /* tokens of the query                             */
  int32_t chunk_len;         /* tokens per retrieved chunk                      */
  int32_t answer_len;        /* tokens an answer-producing call generates       */
  int64_t kv_bytes_per_token;/* K and V of one token over all layers, as held
                                by this GPU (model shape x bytes per element)   */
} rag_request_shape;

typedef struct {
  int32_t method;            /* RAG_STUFF, RAG_MAP_REDUCE_MAP or RAG_MAP_RERANK; -1
                                when nothing fits                                */
  int32_t num_chunks;
  int32_t intermediate_length;  /* 0 unless map_reduce                          */
  int32_t fallback;          /* 1: chosen outside the pruned space (none fitted) */
  int64_t kv_bytes;          /* memory requirement, 2% buffer included          */
} rag_config;

/*
 * Algorithm 1: no joint reasoning -> {map_rerank}; joint reasoning with low
 * complexity -> {stuff}; with high complexity -> {stuff, map_reduce};
 * num_chunks in [pieces, 3 * pieces]; intermediate_length in the summary range.
 * Returns RAG_OK or RAG_ERR_INVALID_ARG (null pointer; flags not 0/1; pieces
 * < 1; empty or non-positive summary range).
 */
rag_status rag_prune_config_space(const rag_query_profile *profile,
                                  rag_config_space *space);

/*
 * KV-cache memory requirement of one configuration, in bytes, with the
 * paper's 2% buffer: tokens * kv_bytes_per_token * 1.02, rounded up (Sec.
 * "Joint configuration-scheduling adaptation").  It is the memory the
 * configuration needs free to start -- the one quantity rag_choose_config
 * compares with the available memory and ranks by.  A call holds its prompt
 * and the tokens it generates.  stuff: one call of num_chunks * chunk_len +
 * query_len prompt tokens; map_rerank: num_chunks calls of chunk_len +
 * query_len, which run together; map_reduce: its largest single call, a
 * mapper (chunk_len + query_len prompt, intermediate_length summary tokens)
 * or the reduce call (num_chunks * intermediate_length + query_len), since
 * its mappers enter the running batch one by one as memory allows and the
 * reduce call runs after them.  -1 for an invalid argument.
 */
int64_t rag_config_kv_bytes(int32_t method, int32_t num_chunks,
                            int32_t intermediate_length,
                            const rag_request_shape *shape);

/*
 * Best-fit choice: among the configurations of the pruned space whose
 * requirement (rag_config_kv_bytes) fits in available_bytes, the one with the
 * highest requirement; ties go to more chunks, then a longer intermediate
 * length, then stuff, map_reduce, map_rerank in that order.  If none fits, a
 * cheaper configuration just outside the space: stuff (joint reasoning) or
 * map_rerank (otherwise) with as many chunks as fit (fallback = 1).  Returns
 * RAG_OK, RAG_NO_FIT (not even one chunk fits: the request waits; *out has
 * method -1) or RAG_ERR_INVALID_ARG.
 */
rag_status rag_choose_config(const rag_query_profile *profile,
                             const rag_request_shape *shape,
                             int64_t available_bytes, rag_config *out);

/* Free and total memory of the current HIP device (hipMemGetInfo), the input
 * of rag_choose_config's available_bytes.  RAG_OK or RAG_ERR_HIP. */
rag_status rag_device_free_memory(size_t *free_bytes, size_t *total_bytes);

/*
 * Group-quantized int4-weight GEMM, the weight format of the served models
 * (Sec. "Setup": both are AWQ-quantized), for the projections and MLP around
 * the attention calls:
 *
 *   y[m, n] = sum_k x[m, k] * (q[k, n] - zeros[g, n]) * scales[g, n],
 *   g = k / group_size.
 *
 * Codes q and zero points are 4-bit unsigned (0..15), one scale and one zero
 * point per group of 128 consecutive k and output column n.  Products and sums
 * run in fp32, y is rounded to bf16 (nearest even).
 *
 * rag_awq_pack_weights (host only) packs codes for the kernel:
 *   q       host uint8 [K, N], each 0..15
 *   packed  host int32 [K / 128, N, 16] (K * N / 8 words): the 64 bytes of
 *           (group g, column n) are contiguous; word 8a + 4b + c holds the
 *           codes of k = 128 g + 8 (4c + 2b + a) + j, j = 0..7, code j in
 *           bits 4 (j / 2) + 16 (j % 2) .. +4
 * Returns RAG_OK, RAG_ERR_INVALID_ARG (null pointer, a code above 15, N or K
 * not positive) or RAG_ERR_UNSUPPORTED (group_size not 128, K or N not a
 * multiple of 128).
 */
rag_status rag_awq_pack_weights(const uint8_t *q, int32_t K, int32_t N,
                                int32_t group_size, int32_t *packed);

/* Bytes of workspace rag_awq_gemm needs (0 for M == 0, invalid shapes, or
 * a small batch that needs none).  Library-internal layout.  M > 64: the
 * group sums of x [K / 128, M] (each as three bf16 pieces in 16 bytes), then,
 * when the output tiles are too few to fill the GPU, fp32 partial outputs
 * [splits, M, N] of a split over the groups.  M <= 64, when the groups are
 * split over workgroups (long K, or too few column blocks to fill the GPU):
 * one arrival counter per column block, then fp32 partial outputs
 * [splits, M, N].  Partials are added in a fixed order, so results do not
 * depend on timing.  For M <= 64 the environment variables RAG_AWQ_SM_NB
 * (16-column blocks per workgroup: 1, 2, 4 or 8) and RAG_AWQ_SM_SPLITS (at
 * least this many splits) override the library's choice, read at each call
 * of this function and of rag_awq_gemm (which must then see the same
 * values); testing knobs: they change the size and the rounding order. */
size_t rag_awq_workspace_size(int32_t M, int32_t N, int32_t K,
                              int32_t group_size);

/*
 *   x        device bf16 [M, K], row-major
 *   qweight  device int32 [K / 128, N, 16] from rag_awq_pack_weights
 *   scales   device bf16 [K / 128, N]
 *   zeros    device uint8 [K / 128, N], each 0..15
 *   y        device bf16 [M, N]; output, written in full
 *   workspace  device, >= rag_awq_workspace_size(M, N, K, group_size) bytes,
 *            256-byte aligned, zero-filled once before its first use: for
 *            small batches split over the weight groups it starts with one
 *            arrival counter per column block, which every call leaves at
 *            zero again.  Overlapping calls must not share it.
 * Returns RAG_OK (M == 0 is a no-op; x and y may then be NULL),
 * RAG_ERR_INVALID_ARG (null pointer, a pointer not 16-byte aligned, negative
 * M, N or K not positive), RAG_ERR_UNSUPPORTED (group_size not 128, K or N not a multiple of
 * 128, M over 4,194,240), RAG_ERR_WORKSPACE or RAG_ERR_HIP.
 */
rag_status rag_awq_gemm(const void *x, const int32_t *qweight,
                        const void *scales, const uint8_t *zeros, void *y,
                        int32_t M, int32_t N, int32_t K, int32_t group_size,
                        void *workspace, size_t workspace_bytes,
                        hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* RAG_ATTN_H */
