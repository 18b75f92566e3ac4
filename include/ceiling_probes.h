/*
 * ceiling_probes.h -- measurement probes for MI355X (gfx950), built into
 * libceiling_probes.so next to librag_attn.so.  They are not part of the
 * attention method: they measure what the hardware gives kernels shaped like
 * the library's, the ceilings its roofline fractions are read against
 * (bench.py --ceilings times them with HIP events).
 *
 * Each call enqueues one kernel on `stream` and returns 0, -1 for an invalid
 * argument, -4 for a launch error.  `sink` is a device buffer of at least
 * 4 * workgroups bytes that the kernel may write (it keeps the reads or the
 * products from being optimised away).
 */
#ifndef RAG_CEILING_PROBES_H
#define RAG_CEILING_PROBES_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Reads num_pages 4096-byte pages of `pool` (device), page i at byte offset
 * 4096 * page_ids[i] (device int32 list, caller-chosen order), with 16-byte
 * loads; each wave keeps four pages (16 KB) in flight.  stream_hint = 1 adds
 * the non-temporal hint to the loads. */
int rag_probe_page_read(const void *pool, const int32_t *page_ids,
                        int64_t num_pages, int32_t workgroups,
                        int32_t stream_hint, void *sink, hipStream_t stream);

/* Reads, for each of num_pages ids, the 4096-byte page at byte offset
 * 4096 * page_ids[i] of k_pool and the one of v_pool (both device), each
 * wave two pairs at a time.  pattern 0: the paged decode kernel's loads (K as
 * its MFMA operand layout, 64 bytes of each of 16 rows per instruction, with
 * the default policy; V as whole 256-byte rows with the non-temporal hint);
 * 1: both as whole rows, default policy; 2: both as whole rows, non-temporal.
 * Counts 8192 bytes per id. */
int rag_probe_kv_page_read(const void *k_pool, const void *v_pool,
                           const int32_t *page_ids, int64_t num_pages,
                           int32_t workgroups, int32_t pattern, void *sink,
                           hipStream_t stream);

/* Reads `bytes` (a multiple of 16) of `buf` contiguously with 16-byte loads;
 * stream_hint = 1 adds the non-temporal hint. */
int rag_probe_stream_read(const void *buf, int64_t bytes, int32_t workgroups,
                          int32_t stream_hint, void *sink, hipStream_t stream);

/* `workgroups` eight-wave workgroups; every wave issues 4 * iters
 * v_mfma_f32_32x32x16_bf16 (32768 FLOP each) into four independent
 * accumulators, with no memory traffic. */
int rag_probe_mfma_loop(int32_t iters, int32_t workgroups, void *sink,
                        hipStream_t stream);

/* `workgroups` eight-wave workgroups, each with two 32 KB LDS stages holding
 * a 64-key K/V tile (d = 128, filled once): every wave runs the prefill
 * kernel's steady slot (32 query rows x 32 keys: QK^T and PV MFMAs, online
 * softmax, LDS operand reads) 2 * iters times, with a workgroup barrier every
 * two slots and no copies.  524288 FLOP per slot and wave (4 x 128 per
 * query-key pair). */
int rag_probe_attn_slot(int32_t iters, int32_t workgroups, void *sink,
                        hipStream_t stream);

/* `workgroups` eight-wave workgroups on the same two LDS tiles, the slot's
 * work split between the two waves of each SIMD: wave w < 4 computes QK^T
 * and the exponentials for 64 query rows (one K read per step for both 32-row
 * blocks) and passes the bf16 weights through LDS to wave w + 4, which runs
 * PV for the 64 rows; a workgroup barrier per 32-key block, iters blocks.
 * 1048576 FLOP per block and wave pair. */
int rag_probe_attn_pair(int32_t iters, int32_t workgroups, void *sink,
                        hipStream_t stream);

/* The same instruction mix as rag_probe_attn_slot with K/V operands in
 * registers (no LDS): 2 * iters slots of 16 MFMAs and the softmax vector work of
 * 32 x 32 scores per wave. */
int rag_probe_softmax_mfma(int32_t iters, int32_t workgroups, void *sink,
                           hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* RAG_CEILING_PROBES_H */
