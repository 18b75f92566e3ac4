/*
 * fp64 CPU oracle for the RAG-synthesis attention path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's
 * CPU-baseline leg may load this library.  It shares no code, header or
 * constant with the GPU library and never calls it.
 *
 * What it computes is the plain definition of scaled-dot-product attention
 * (softmax(q k^T * scale) v) over the tokens a synthesis call feeds the LLM:
 *   - the synthesis step (Sec. "RAG systems and configurations") turns the
 *     retrieved chunks and the query into one prompt (stuff) or one prompt per
 *     chunk (map_reduce mappers, map_rerank); the LLM then prefills that prompt
 *     and decodes the answer;
 *   - the serving engine keeps the KV cache in fixed-size pages addressed by a
 *     per-sequence block table (the paged-attention engine named in Sec.
 *     "Implementation") and mixes running decodes with chunked prefills in one
 *     batch (Sec. "Joint configuration-scheduling adaptation").
 * The attention formula itself is not printed in the paper; it is the standard
 * transformer attention of the served models.  Readings used where the paper
 * is silent:
 *   - scale is a caller argument (1/sqrt(d) in every workload);
 *   - grouped-query heads: q head h reads kv head floor(h * Hkv / Hq);
 *   - causal masking is bottom-right aligned: with nq query rows and nk keys,
 *     query row i sees keys j <= (nk - nq) + i (chunked prefill of a suffix);
 *   - paged keys: logical key j of sequence s lives in
 *     cache[block_table[s][j / bs]][g][j % bs][:].
 *
 * Every value is fp64; bf16 inputs are widened exactly by the Python wrapper
 * before they reach this file.  Each output row is computed in two passes
 * (maximum, then exponentials and sums) straight from the definition
 *   m = max_j s_j,  Z = sum_j exp(s_j - m),
 *   o = sum_j exp(s_j - m) v_j / Z,  lse = m + ln Z.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>

/* One query row against an explicit list of visible key/value rows.
 * krow[j], vrow[j] point at d-element fp64 rows.  p (nullable) receives the
 * nvis softmax weights in key order. */
void oracle_attend_row(const double *q, const double *const *krow,
                       const double *const *vrow, int32_t nvis, int32_t d,
                       double scale, double *o, double *lse, double *p) {
  double *s = (double *)malloc(sizeof(double) * (size_t)(nvis > 0 ? nvis : 1));
  double m = -INFINITY;
  for (int32_t j = 0; j < nvis; ++j) {
    double dot = 0.0;
    for (int32_t c = 0; c < d; ++c) dot += q[c] * krow[j][c];
    s[j] = dot * scale;
    if (s[j] > m) m = s[j];
  }
  double z = 0.0;
  for (int32_t j = 0; j < nvis; ++j) {
    s[j] = exp(s[j] - m);
    z += s[j];
  }
  for (int32_t c = 0; c < d; ++c) o[c] = 0.0;
  for (int32_t j = 0; j < nvis; ++j) {
    const double w = s[j] / z;
    if (p) p[j] = w;
    for (int32_t c = 0; c < d; ++c) o[c] += w * vrow[j][c];
  }
  if (lse) *lse = m + log(z);
  free(s);
}

/* Keys visible to query row i of a sequence with nq rows and nk keys. */
static int32_t visible_keys(int32_t i, int32_t nq, int32_t nk, int32_t causal) {
  if (!causal) return nk;
  return (nk - nq) + i + 1;
}

/*
 * Packed variable-length attention (prefill).
 *   q [Tq, hq, d], k and v [Tk, hkv, d], o [Tq, hq, d]; lse [hq, Tq] or NULL.
 *   Sequence s owns q rows [cu_q[s], cu_q[s+1]) and k/v rows
 *   [cu_k[s], cu_k[s+1]).
 */
void oracle_attention_varlen(const double *q, const double *k, const double *v,
                             double *o, double *lse, const int32_t *cu_q,
                             const int32_t *cu_k, int32_t num_seqs, int32_t hq,
                             int32_t hkv, int32_t d, double scale,
                             int32_t causal) {
  int32_t tq = cu_q[num_seqs];
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
  for (int32_t s = 0; s < num_seqs; ++s) {
    for (int32_t h = 0; h < hq; ++h) {
      const int32_t g = (int32_t)(((int64_t)h * hkv) / hq);
      const int32_t q0 = cu_q[s], nq = cu_q[s + 1] - cu_q[s];
      const int32_t k0 = cu_k[s], nk = cu_k[s + 1] - cu_k[s];
      const double **kr = (const double **)malloc(sizeof(double *) * (size_t)(nk > 0 ? nk : 1));
      const double **vr = (const double **)malloc(sizeof(double *) * (size_t)(nk > 0 ? nk : 1));
      for (int32_t j = 0; j < nk; ++j) {
        kr[j] = k + ((size_t)(k0 + j) * hkv + g) * d;
        vr[j] = v + ((size_t)(k0 + j) * hkv + g) * d;
      }
      for (int32_t i = 0; i < nq; ++i) {
        const size_t row = (size_t)(q0 + i);
        double *lp = lse ? lse + (size_t)h * tq + row : NULL;
        oracle_attend_row(q + (row * hq + h) * d, kr, vr,
                          visible_keys(i, nq, nk, causal), d, scale,
                          o + (row * hq + h) * d, lp, NULL);
      }
      free(kr);
      free(vr);
    }
  }
}

/*
 * Attention against a paged KV cache (decode, chunked prefill, or both in one
 * batch).
 *   q [Tq, hq, d]; sequence s owns q rows [cu_q[s], cu_q[s+1]), or the single
 *   row s when cu_q is NULL.  k_cache and v_cache [num_blocks, hkv, bs, d];
 *   block_tables [num_seqs, max_blocks]; kv_lens [num_seqs] counts every key
 *   of the sequence including the ones belonging to its own query rows.
 *   Masking is causal, bottom-right aligned.  o [Tq, hq, d]; lse [hq, Tq] or
 *   NULL.
 */
void oracle_attention_paged(const double *q, const double *k_cache,
                            const double *v_cache, double *o, double *lse,
                            const int32_t *block_tables, const int32_t *kv_lens,
                            const int32_t *cu_q, int32_t num_seqs,
                            int32_t max_blocks, int32_t bs, int32_t hq,
                            int32_t hkv, int32_t d, double scale) {
  int32_t tq = cu_q ? cu_q[num_seqs] : num_seqs;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
  for (int32_t s = 0; s < num_seqs; ++s) {
    for (int32_t h = 0; h < hq; ++h) {
      const int32_t g = (int32_t)(((int64_t)h * hkv) / hq);
      const int32_t q0 = cu_q ? cu_q[s] : s;
      const int32_t nq = cu_q ? cu_q[s + 1] - cu_q[s] : 1;
      const int32_t nk = kv_lens[s];
      const double **kr = (const double **)malloc(sizeof(double *) * (size_t)(nk > 0 ? nk : 1));
      const double **vr = (const double **)malloc(sizeof(double *) * (size_t)(nk > 0 ? nk : 1));
      for (int32_t j = 0; j < nk; ++j) {
        const int32_t blk = block_tables[(size_t)s * max_blocks + j / bs];
        const size_t off = (((size_t)blk * hkv + g) * bs + (size_t)(j % bs)) * d;
        kr[j] = k_cache + off;
        vr[j] = v_cache + off;
      }
      for (int32_t i = 0; i < nq; ++i) {
        const size_t row = (size_t)(q0 + i);
        double *lp = lse ? lse + (size_t)h * tq + row : NULL;
        oracle_attend_row(q + (row * hq + h) * d, kr, vr,
                          visible_keys(i, nq, nk, 1), d, scale,
                          o + (row * hq + h) * d, lp, NULL);
      }
      free(kr);
      free(vr);
    }
  }
}

/*
 * Selected query rows of one sequence, for workloads too large to evaluate in
 * full.  q_rows [n, d] holds the query vectors, row_idx[n] their row index
 * within the sequence (0-based, of nq rows) and heads[n] their q head; k and
 * v [nk, hkv, d] are that sequence's keys and values.  o_rows [n, d] and
 * lse_rows [n] receive the results.
 */
void oracle_attention_seq_rows(const double *q_rows, const double *k,
                               const double *v, int32_t nq, int32_t nk,
                               int32_t hq, int32_t hkv, int32_t d,
                               double scale, int32_t causal,
                               const int32_t *row_idx, const int32_t *heads,
                               int32_t n, double *o_rows, double *lse_rows) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int32_t r = 0; r < n; ++r) {
    const int32_t g = (int32_t)(((int64_t)heads[r] * hkv) / hq);
    const double **kr = (const double **)malloc(sizeof(double *) * (size_t)(nk > 0 ? nk : 1));
    const double **vr = (const double **)malloc(sizeof(double *) * (size_t)(nk > 0 ? nk : 1));
    for (int32_t j = 0; j < nk; ++j) {
      kr[j] = k + ((size_t)j * hkv + g) * d;
      vr[j] = v + ((size_t)j * hkv + g) * d;
    }
    oracle_attend_row(q_rows + (size_t)r * d, kr, vr,
                      visible_keys(row_idx[r], nq, nk, causal), d, scale,
                      o_rows + (size_t)r * d, lse_rows + r, NULL);
    free(kr);
    free(vr);
  }
}
