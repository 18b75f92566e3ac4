// One decode unit on gfx950: a workgroup of W waves (four, or eight inside the
// mixed launch) attends the query row
// of every q head of one GQA group (one decode token of one sequence) to a
// contiguous range of pages of that sequence's paged KV cache.
//
// Method: paged KV (PagedAttention) read through the block table, split-KV
// with a log-sum-exp merge of the partial results (Flash-Decoding), online
// softmax in fp32.  Layout choices for CDNA4:
//   * every K/V byte of the range is read once, for all G heads of the group,
//     with 16-byte loads; the W waves take interleaved steps of NP pages,
//     so at any time they stream neighbouring pages; the V loads (each
//     instruction covers four whole 256-byte rows) carry the non-temporal
//     hint, as nothing of a decode step's pages is read again in the launch;
//     the K loads (64 bytes of each of 16 rows per instruction, two
//     instructions per 128-byte line) do not, as that made them slower;
//   * both products run on v_mfma_f32_16x16x32_bf16 with the G query heads as
//     the N dimension (padded to 16): S^T = K Q^T straight from registers,
//     then O^T = V^T P^T with the V rows staged row-major in a per-wave LDS
//     slice and read back as V^T fragments by the transposing LDS read;
//   * one register set per step is refilled as soon as it has been consumed,
//     so the next step's pages are in flight while the current one computes;
//   * the W waves' states are merged through LDS; a unit that covers only
//     part of its sequence (a split) writes a normalised partial output and
//     its log-sum-exp, and the last split of the sequence to finish merges
//     all of them in the same kernel.
#pragma once

#include "common.h"

namespace rag {

// Where a unit's result goes.  h0 is the first q head of the group.
struct DecodeOut {
  bf16_t* o;            // final output row of head h0
  float* part_o;        // partials of head h0: [head][split][D] (n_sp > 1)
  float* part_lse;      // [head][split]
  int* arrival;         // arrival counter of this (sequence, kv head)
  int sp, n_sp, num_splits;
};

// Per wave: attend the wave's steps of the page range.  Leaves, per lane
// (head l16, lane group gq), the unnormalised O^T accumulators, the head's
// sum of weights l (already reduced over the lane groups) and the reference
// maximum m_used (raw score units).
//
// kAppend: key kv_len - 1 is the step's new token, whose K and V rows are
// k_new and v_new (this kv head's rows) rather than the cache: the lanes that
// would load that slot read them there instead (the cache slot is written in
// the same launch, see decode_unit).
template <int D, int NP, bool kAppend = false>
__device__ __forceinline__ void decode_wave(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    size_t block_stride, const int32_t* __restrict__ table, int kv_len, int group,
    int p_first, int p_end, int p_stride, float scale, bf16_t* __restrict__ vt,
    f32x4 (&oacc)[D / 16], float& m_used, float& l, const bf16_t* __restrict__ k_new = nullptr,
    const bf16_t* __restrict__ v_new = nullptr) {
  static_assert(NP % 2 == 0, "pages are consumed in pairs (32 keys per MFMA)");
  using L = DecLds<D, NP>;
  constexpr int kKs = D / 32;   // k-steps over d for S^T
  constexpr int kDt = D / 16;   // 16-row d tiles of O^T
  const int lane = threadIdx.x & 63;
  const int l16 = lane & 15, gq = lane >> 4;

  // Q^T fragments: lane holds head l16, d = 32*ks + 8*gq .. +8.
  bf16x8 qf[kKs];
#pragma unroll
  for (int ks = 0; ks < kKs; ++ks) {
    u32x4 z = {0, 0, 0, 0};
    qf[ks] = as_bf16x8(l16 < group ? load16(q + (size_t)l16 * D + ks * 32 + gq * 8) : z);
  }
#pragma unroll
  for (int dt = 0; dt < kDt; ++dt) oacc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const float c = scale * kLog2e;
  const float tau = kRescaleLog2 / c;
  m_used = -INFINITY;
  l = 0.f;

  //   kr[j]: K rows of page j as the MFMA A operand (key l16, d chunk 4*ks+gq)
  //   vr[j]: V rows of page j (keys 4*gq + t, d chunk l16) for the LDS slice
  u32x4 kr[NP][kKs], vr[NP][4];
  constexpr int kVch = D / 8;                  // 16-byte chunks per V row
  // Block ids of the wave's next 64 / NP steps, one per lane (lane NP*k + j
  // holds page j of step k), fetched with one vector load so that issuing a
  // step's loads never waits on a scalar block-table read.
  constexpr int kStepsPerFetch = kWave / NP;
  int ids = 0, ids_base = p_first;
  auto fetch_ids = [&](int p_from) {
    const int pg = p_from + (lane / NP) * p_stride + lane % NP;
    ids = pg < p_end ? table[pg] : 0;
    ids_base = p_from;
  };
  auto issue_loads = [&](int p0) {
    const int k = (p0 - ids_base) / p_stride;
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      const int id = __builtin_amdgcn_readlane(ids, k * NP + (p0 + j < p_end ? j : 0));
      const size_t base = (size_t)id * block_stride;
      if constexpr (kAppend) {
        const int key0 = 16 * (p0 + j);
        const bf16_t* kp = key0 + l16 == kv_len - 1 ? k_new : kc + base + (size_t)l16 * D;
#pragma unroll
        for (int ks = 0; ks < kKs; ++ks) kr[j][ks] = load16(kp + ks * 32 + gq * 8);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const bf16_t* vp =
              key0 + 4 * gq + t == kv_len - 1 ? v_new : vc + base + (size_t)(4 * gq + t) * D;
          vr[j][t] = load16_stream(vp + (l16 % kVch) * 8);
        }
      } else {
#pragma unroll
        for (int ks = 0; ks < kKs; ++ks)
          kr[j][ks] = load16(kc + base + (size_t)l16 * D + ks * 32 + gq * 8);
#pragma unroll
        for (int t = 0; t < 4; ++t)
          vr[j][t] = load16_stream(vc + base + (size_t)(4 * gq + t) * D + (l16 % kVch) * 8);
      }
    }
  };

  // transposing-read source: row 4*gq + l16/4, d 4*(l16%4) of a 16-d tile
  const int tr_off = (4 * gq + (l16 >> 2)) * L::kStrV + 4 * (l16 & 3);

  if (p_first < p_end) {
    fetch_ids(p_first);
    issue_loads(p_first);
  }
  for (int p0 = p_first; p0 < p_end; p0 += p_stride) {
    // ---- V rows into this wave's LDS slice (row 16*j + key of page j).  Rows
    // of keys past kv_len (tail slots) or of pages past the range are zeroed
    // so that whatever the pool holds there cannot reach the output. ---------
#pragma unroll
    for (int j = 0; j < NP; ++j) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int key = 16 * (p0 + j) + 4 * gq + t;
        const bool valid = p0 + j < p_end && key < kv_len;
        u32x4 z = {0, 0, 0, 0};
        if (l16 < kVch)
          *reinterpret_cast<u32x4*>(vt + (16 * j + 4 * gq + t) * L::kStrV + l16 * 8) =
              valid ? vr[j][t] : z;
      }
    }
    // ---- S^T = K Q^T: 16 keys x 16 heads per page --------------------------
    f32x4 sc[NP];
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      sc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < kKs; ++ks) sc[j] = mfma16(as_bf16x8(kr[j][ks]), qf[ks], sc[j]);
    }
    // ---- next step's loads go out now ---------------------------------------
    if (p0 + p_stride < p_end) {
      if ((p0 + p_stride - ids_base) / p_stride == kStepsPerFetch) fetch_ids(p0 + p_stride);
      issue_loads(p0 + p_stride);
    }

    // ---- mask and online softmax ---------------------------------------------
    float tmax = -INFINITY;
#pragma unroll
    for (int j = 0; j < NP; ++j) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int key = 16 * (p0 + j) + 4 * gq + t;
        if (p0 + j >= p_end || key >= kv_len) sc[j][t] = -INFINITY;
        tmax = fmaxf(tmax, sc[j][t]);
      }
    }
    tmax = fmaxf(tmax, wave_xor(tmax, 16));
    tmax = fmaxf(tmax, wave_xor(tmax, 32));
    if (wave_any(tmax > m_used + tau)) {
      const float m_new = fmaxf(m_used, tmax);
      const float alpha = (m_used == -INFINITY) ? 0.f : fast_exp2((m_used - m_new) * c);
      l *= alpha;
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt) oacc[dt] *= alpha;
      m_used = m_new;
    }
    const float mref = (m_used == -INFINITY) ? 0.f : m_used * c;
    bf16x8 pfrag[NP / 2];
#pragma unroll
    for (int pp = 0; pp < NP / 2; ++pp) {
      float pv[8];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        pv[t] = fast_exp2(fmaf(sc[2 * pp][t], c, -mref));
        pv[4 + t] = fast_exp2(fmaf(sc[2 * pp + 1][t], c, -mref));
        l += pv[t] + pv[4 + t];
      }
      pfrag[pp] = to_bf16x8(pv[0], pv[1], pv[2], pv[3], pv[4], pv[5], pv[6], pv[7]);
    }

    wave_lds_sync();
    // ---- O^T += V^T P^T ------------------------------------------------------
    // Pair pp (pages 2pp, 2pp+1): A operand slot 8*gq + t holds key 4*gq + t
    // of page 2pp (t < 4) or page 2pp+1 (t >= 4) at d = 16*dt + l16 -- two
    // transposing reads whose 16-lane groups each cover 4 rows x 16 d.
#pragma unroll
    for (int pp = 0; pp < NP / 2; ++pp) {
      const bf16_t* v0 = vt + 32 * pp * L::kStrV + tr_off;
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt) {
        const bf16x8 a = join_bf16x8(lds_read_tr4(v0 + 16 * dt),
                                     lds_read_tr4(v0 + 16 * L::kStrV + 16 * dt));
        oacc[dt] = mfma16(a, pfrag[pp], oacc[dt]);
      }
    }
    wave_lds_sync();
  }
  l += wave_xor(l, 16);
  l += wave_xor(l, 32);
}

// Merge of the n_sp split partials of the q heads assigned to this wave (h =
// wave, wave + W, ...), in split order.  Lane sp holds split sp's weight; the
// partial rows are read with device-coherent loads, 16 splits at a time, each
// lane owning D/64 consecutive output values.
template <int D, int W>
__device__ __forceinline__ void merge_splits(const DecodeOut& out, int group) {
  constexpr int kPer = D / 64;                 // 2 (D = 128) or 1 (D = 64)
  constexpr int kBatch = 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int h = wave; h < group; h += W) {
    const float* pl = out.part_lse + (size_t)h * out.num_splits;
    const float* po = out.part_o + (size_t)h * out.num_splits * D + lane * kPer;
    const float lse = lane < out.n_sp ? load_coherent(pl + lane) : -INFINITY;
    float mx = lse;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) mx = fmaxf(mx, wave_xor(mx, m));
    const float w = (lse == -INFINITY) ? 0.f : fast_exp2((lse - mx) * kLog2e);
    float den = w;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) den += wave_xor(den, m);
    float acc[kPer];
#pragma unroll
    for (int e = 0; e < kPer; ++e) acc[e] = 0.f;
    for (int s0 = 0; s0 < out.n_sp; s0 += kBatch) {
      float x[kBatch][kPer];
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int sp = s0 + b < out.n_sp ? s0 + b : s0;
#pragma unroll
        for (int e = 0; e < kPer; ++e) x[b][e] = load_coherent(po + (size_t)sp * D + e);
      }
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const float wb = __shfl(w, s0 + b < out.n_sp ? s0 + b : 0, kWave);
        if (s0 + b < out.n_sp) {
#pragma unroll
          for (int e = 0; e < kPer; ++e) acc[e] += wb * x[b][e];
        }
      }
    }
    const float inv = den > 0.f ? 1.f / den : 0.f;
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
      const __bf16 b = (__bf16)(acc[e] * inv);
      out.o[(size_t)h * D + lane * kPer + e] = __builtin_bit_cast(bf16_t, b);
    }
  }
}

// Bytes of LDS the merge of W waves needs (it reuses the V slices).
template <int D, int W>
constexpr int dec_merge_bytes() {
  return (W * 16 * D + 2 * W * 16 + 1) * 4;
}

// The whole unit: the workgroup's W waves cover the page range
// [p_begin, p_end) in interleaved steps of NP pages, merge through LDS and
// write either the final rows (n_sp == 1) or this split's partial rows; the
// last split of the row to arrive then merges all partials.
//
// kAppend: the unit whose range holds the last page also stores the new
// token's K and V rows (k_new, v_new) into its cache slot, key kv_len - 1 of
// the block table.  No unit of this launch reads that slot from the cache.
template <int D, int NP, int W, bool kAppend = false>
__device__ __forceinline__ void decode_unit(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    size_t block_stride, const int32_t* __restrict__ table, int kv_len, int group,
    int p_begin, int p_end, float scale, const DecodeOut& out, bf16_t* __restrict__ lds,
    const bf16_t* __restrict__ k_new = nullptr, const bf16_t* __restrict__ v_new = nullptr) {
  using L = DecLds<D, NP, W>;
  static_assert(dec_merge_bytes<D, W>() <= L::kBytes, "merge area must fit in the V slices");
  constexpr int kDt = D / 16;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int l16 = lane & 15, gq = lane >> 4;

  if constexpr (kAppend) {
    constexpr int kCh = D / 8;
    if (wave == 0 && p_end == (kv_len + 15) >> 4 && lane < 2 * kCh) {
      const int key = kv_len - 1;
      const size_t dst = (size_t)table[key >> 4] * block_stride + (size_t)(key & 15) * D +
                         (lane % kCh) * 8;
      const bf16_t* src = (lane < kCh ? k_new : v_new) + (lane % kCh) * 8;
      bf16_t* cache = const_cast<bf16_t*>(lane < kCh ? kc : vc);
      *reinterpret_cast<u32x4*>(cache + dst) = load16(src);
    }
  }
  f32x4 oacc[kDt];
  float m_used, l;
  decode_wave<D, NP, kAppend>(q, kc, vc, block_stride, table, kv_len, group,
                              p_begin + wave * NP, p_end, W * NP, scale,
                              lds + wave * L::kElemsWave, oacc, m_used, l, k_new, v_new);

  // ---- merge the W waves through LDS (reusing the V slices) -------------
  // floats: O [wave][16 heads][D], then m [wave][16], then l [wave][16]
  float* mo = reinterpret_cast<float*>(lds);
  float* mm = mo + W * 16 * D;
  float* ml = mm + W * 16;
  __syncthreads();
  if (l16 < group) {
#pragma unroll
    for (int dt = 0; dt < kDt; ++dt)
      *reinterpret_cast<f32x4*>(mo + (wave * 16 + l16) * D + 16 * dt + 4 * gq) = oacc[dt];
    if (gq == 0) {
      mm[wave * 16 + l16] = m_used;
      ml[wave * 16 + l16] = l;
    }
  }
  __syncthreads();
  const float c = scale * kLog2e;
  constexpr int kPer = D / 64;
  for (int h = wave; h < group; h += W) {
    float m = -INFINITY;
#pragma unroll
    for (int w = 0; w < W; ++w) m = fmaxf(m, mm[w * 16 + h]);
    float den = 0.f, acc[kPer];
#pragma unroll
    for (int e = 0; e < kPer; ++e) acc[e] = 0.f;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const float mw = mm[w * 16 + h];
      const float f = (mw == -INFINITY) ? 0.f : fast_exp2((mw - m) * c);
      den += f * ml[w * 16 + h];
#pragma unroll
      for (int e = 0; e < kPer; ++e) acc[e] += f * mo[(w * 16 + h) * D + lane * kPer + e];
    }
    const float inv = den > 0.f ? 1.f / den : 0.f;
    if (out.n_sp <= 1) {
#pragma unroll
      for (int e = 0; e < kPer; ++e) {
        const __bf16 b = (__bf16)(acc[e] * inv);
        out.o[(size_t)h * D + lane * kPer + e] = __builtin_bit_cast(bf16_t, b);
      }
    } else {
      // Partials may be merged by a workgroup on another XCD: coherent stores.
      float* prow = out.part_o + ((size_t)h * out.num_splits + out.sp) * D + lane * kPer;
#pragma unroll
      for (int e = 0; e < kPer; ++e) store_coherent(prow + e, acc[e] * inv);
      if (lane == 0)
        store_coherent(out.part_lse + (size_t)h * out.num_splits + out.sp,
                       den > 0.f ? m * scale + __logf(den) : -INFINITY);
    }
  }
  if (out.n_sp <= 1) return;

  // ---- arrival: the last split of this (sequence, kv head) merges ----------
  // Every partial has gone out with device-coherent stores; once they have
  // completed, one arrival is counted with a device-scope atomic.  The
  // workgroup that sees the final count reads all partials with
  // device-coherent loads and resets the counter, so the workspace is all-zero
  // between calls.
  wait_all_memory();
  __syncthreads();
  int* flag = reinterpret_cast<int*>(ml + W * 16);
  if (threadIdx.x == 0)
    *flag = __hip_atomic_fetch_add(out.arrival, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (*flag != out.n_sp - 1) return;
  merge_splits<D, W>(out, group);
  if (threadIdx.x == 0)
    __hip_atomic_store(out.arrival, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace rag
