// One decode unit on gfx950: a single wave attends the query rows of all q
// heads of one GQA group (one decode token of one sequence) to a contiguous
// range of pages of that sequence's paged KV cache.
//
// Method: paged KV (PagedAttention) read through the block table, split-KV
// with a log-sum-exp merge of the partial results (Flash-Decoding), online
// softmax in fp32.  Layout choices for CDNA4:
//   * every K/V byte of the range is read once, for all G heads of the
//     group, with 16-byte loads; for each key the four lane groups of a load
//     instruction read 64 contiguous bytes of that key's row;
//   * both products run on v_mfma_f32_16x16x32_bf16 with the G query heads as
//     the N dimension (padded to 16): S^T = K Q^T straight from registers,
//     then O^T = V^T P^T with the V rows staged row-major in a per-wave LDS
//     slice and read back as V^T fragments by the transposing LDS read;
//   * two pages (32 keys) per step; the next step's pages are loaded while
//     the current step computes.
#pragma once

#include "common.h"

namespace rag {

// Orders LDS traffic between the lanes of one wave (a wave-scope fence plus
// a scheduling barrier; no workgroup barrier is needed).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

struct DecodeOut {
  bf16_t* o;          // final output of head 0 of the group (null when split)
  float* part_o;      // partial output of head 0 (null when not split)
  float* part_lse;    // partial log-sum-exp of head 0
  int head_stride_part;  // floats between consecutive heads in part_o (lse: / D)
};

template <int D>
__device__ __forceinline__ void decode_unit(
    const bf16_t* __restrict__ q,          // query row of head 0 of the group
    const bf16_t* __restrict__ kc,         // k cache at (block 0, kv head)
    const bf16_t* __restrict__ vc,
    size_t block_stride,                   // elements between blocks
    const int32_t* __restrict__ table,     // block table row of the sequence
    int kv_len, int group, int p_begin, int p_end, float scale,
    const DecodeOut& out, bf16_t* __restrict__ vt /* per-wave LDS tile */) {
  using L = DecLds<D>;
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
  f32x4 oacc[kDt];
#pragma unroll
  for (int dt = 0; dt < kDt; ++dt) oacc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const float c = scale * kLog2e;
  const float tau = kRescaleLog2 / c;
  float m_used = -INFINITY;
  float l = 0.f;

  // Register staging for one step (two pages):
  //   ka/kb: K rows as the MFMA A operand (key l16, d chunk 4*ks + gq)
  //   va/vb: V rows (keys 4*gq + t, d chunk l16) for the LDS slice
  u32x4 ka[kKs], kb[kKs], va[4], vb[4];
  auto load_step = [&](int p) {
    const bool has_b = p + 1 < p_end;
    const size_t ba = (size_t)table[p] * block_stride;
    const size_t bb = has_b ? (size_t)table[p + 1] * block_stride : ba;
#pragma unroll
    for (int ks = 0; ks < kKs; ++ks) {
      ka[ks] = load16(kc + ba + (size_t)l16 * D + ks * 32 + gq * 8);
      kb[ks] = load16(kc + bb + (size_t)l16 * D + ks * 32 + gq * 8);
    }
    if constexpr (D == 128) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        va[t] = load16(vc + ba + (size_t)(4 * gq + t) * D + l16 * 8);
        vb[t] = load16(vc + bb + (size_t)(4 * gq + t) * D + l16 * 8);
      }
    } else {
      // D == 64: 8 chunks per row; lanes l16 and l16 + 8 load the same chunk
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        va[t] = load16(vc + ba + (size_t)(4 * gq + t) * D + (l16 & 7) * 8);
        vb[t] = load16(vc + bb + (size_t)(4 * gq + t) * D + (l16 & 7) * 8);
      }
    }
  };

  // transposing-read source: row 4*gq + l16/4, d 4*(l16%4) of a 16-d tile
  const int tr_off = (4 * gq + (l16 >> 2)) * L::kStrV + 4 * (l16 & 3);

  if (p_begin < p_end) load_step(p_begin);
  for (int p = p_begin; p < p_end; p += 2) {
    const bool has_b = p + 1 < p_end;
    // ---- S^T = K Q^T: 16 keys x 16 heads per page --------------------------
    f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < kKs; ++ks) {
      sa = mfma16(as_bf16x8(ka[ks]), qf[ks], sa);
      sb = mfma16(as_bf16x8(kb[ks]), qf[ks], sb);
    }
    // V rows of keys past kv_len (tail slots) or of a missing second page are
    // zeroed so that whatever the pool holds there cannot reach the output.
    const int key_a = 16 * p + 4 * gq;       // this lane's first score key, page A
    const int key_b = key_a + 16;
    u32x4 z = {0, 0, 0, 0};
    u32x4 wa[4], wb[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      wa[t] = (key_a + t < kv_len) ? va[t] : z;
      wb[t] = (has_b && key_b + t < kv_len) ? vb[t] : z;
    }
    // Prefetch the next step (registers ka/kb/va/vb are free again).
    if (p + 2 < p_end) load_step(p + 2);

    // ---- mask and online softmax ---------------------------------------------
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (key_a + t >= kv_len) sa[t] = -INFINITY;
      if (!has_b || key_b + t >= kv_len) sb[t] = -INFINITY;
    }
    float tmax = fmaxf(fmaxf(fmaxf(sa[0], sa[1]), fmaxf(sa[2], sa[3])),
                       fmaxf(fmaxf(sb[0], sb[1]), fmaxf(sb[2], sb[3])));
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
    float pa[4], pbv[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      pa[t] = fast_exp2(fmaf(sa[t], c, -mref));
      pbv[t] = fast_exp2(fmaf(sb[t], c, -mref));
      l += pa[t] + pbv[t];
    }
    const bf16x8 pfrag = to_bf16x8(pa[0], pa[1], pa[2], pa[3], pbv[0], pbv[1], pbv[2], pbv[3]);

    // ---- V rows of both pages into this wave's LDS slice, row-major:
    // rows 0..15 page A, rows 16..31 page B ------------------------------------
    if (D == 128 || l16 < 8) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        *reinterpret_cast<u32x4*>(vt + (4 * gq + t) * L::kStrV + l16 * 8) = wa[t];
        *reinterpret_cast<u32x4*>(vt + (16 + 4 * gq + t) * L::kStrV + l16 * 8) = wb[t];
      }
    }
    wave_lds_sync();
    // ---- O^T += V^T P^T ------------------------------------------------------
    // A operand of d-tile dt: slot 8*gq + t holds key 4*gq + t of page A
    // (t < 4) or page B (t >= 4) at d = 16*dt + l16 -- two transposing reads
    // whose 16-lane groups each cover 4 rows x 16 d of one page.
#pragma unroll
    for (int dt = 0; dt < kDt; ++dt) {
      const bf16x8 a = join_bf16x8(lds_read_tr4(vt + tr_off + 16 * dt),
                                   lds_read_tr4(vt + 16 * L::kStrV + tr_off + 16 * dt));
      oacc[dt] = mfma16(a, pfrag, oacc[dt]);
    }
    wave_lds_sync();
  }

  // ---- combine the four lane groups' sums and write ---------------------------
  l += wave_xor(l, 16);
  l += wave_xor(l, 32);
  const float inv = l > 0.f ? 1.f / l : 0.f;
  if (l16 < group) {
    if (out.o != nullptr) {
      bf16_t* orow = out.o + (size_t)l16 * D;
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt) {
        const bf16x4 w = to_bf16x4(oacc[dt][0] * inv, oacc[dt][1] * inv,
                                   oacc[dt][2] * inv, oacc[dt][3] * inv);
        *reinterpret_cast<bf16x4*>(orow + 16 * dt + 4 * gq) = w;
      }
    } else {
      float* prow = out.part_o + (size_t)l16 * out.head_stride_part;
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt)
        *reinterpret_cast<f32x4*>(prow + 16 * dt + 4 * gq) = oacc[dt] * inv;
      if (gq == 0)
        out.part_lse[(size_t)l16 * (out.head_stride_part / D)] =
            l > 0.f ? m_used * scale + __logf(l) : -INFINITY;
    }
  }
}

}  // namespace rag
