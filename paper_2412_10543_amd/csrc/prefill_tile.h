// Causal (or full) attention of one query tile against the keys of its
// sequence, for gfx950: four waves of 32 rows each, covering up to four q heads
// of one GQA group (which share every K/V tile) times the row blocks of the
// tile.
//
// Method: exact tiled attention with an online softmax (FlashAttention's
// forward pass; the running-max rescaling of Milakov & Gimelshein), laid out
// for CDNA4:
//   * 4 or 8 waves, each owning 32 query rows of one head; the wave keeps its Q
//     rows in registers as the B operand of v_mfma_f32_32x32x16_bf16; K/V
//     tiles are shared by all heads of the group in the workgroup;
//   * K/V tiles of 64 keys are staged through LDS row-major ([key][d]),
//     double-buffered, with one barrier per tile; the global loads of the
//     next one or two tiles are in flight while a tile is computed;
//   * scores are computed transposed, S^T = K Q^T, so each lane owns one query
//     row and its scores already sit where the B operand of O^T = V^T P^T
//     needs them; the matching V^T A operand comes straight from the
//     row-major V tile through the transposing LDS read (ds_read_b64_tr_b16),
//     so no data is shuffled between the two products and nothing is
//     transposed on the way into LDS;
//   * softmax statistics in fp32 with exp2 and the scale folded into one
//     FMA; the reference maximum is moved lazily (only when a score exceeds
//     it by 2^8), which keeps rescales of the output off the common path;
//   * masking only on tiles that cross the causal diagonal or the sequence
//     end; tiles fully above the diagonal are skipped per wave.
#pragma once

#include "common.h"

namespace rag {

// K/V rows of one (sequence, kv head) stored densely: token j at k + j*stride.
struct DenseKV {
  const bf16_t* k;
  const bf16_t* v;
  size_t stride;
  __device__ __forceinline__ const bf16_t* krow(int j) const { return k + (size_t)j * stride; }
  __device__ __forceinline__ const bf16_t* vrow(int j) const { return v + (size_t)j * stride; }
};

// K/V rows of one (sequence, kv head) in a paged cache: token j lives in
// physical block table[j / 16], slot j % 16.  k and v already point at the kv
// head inside block 0; block_stride is the distance between blocks.
template <int D>
struct PagedKV {
  const bf16_t* k;
  const bf16_t* v;
  const int32_t* table;
  size_t block_stride;
  __device__ __forceinline__ size_t off(int j) const {
    return (size_t)table[j >> 4] * block_stride + (size_t)(j & 15) * D;
  }
  __device__ __forceinline__ const bf16_t* krow(int j) const { return k + off(j); }
  __device__ __forceinline__ const bf16_t* vrow(int j) const { return v + off(j); }
};

// q, o and lse point at row 0 of the sequence for this wave's head; the
// workgroup (W waves) covers rows [q0, q0 + wg_rows) and this wave rows
// [r0, r0 + 32).  DEPTH = number of K/V tiles whose global loads are in
// flight while a tile is computed (1 or 2).
template <int D, int W, int DEPTH, class KV>
__device__ __forceinline__ void prefill_tile(
    const bf16_t* __restrict__ q, size_t q_stride,
    bf16_t* __restrict__ o, size_t o_stride,
    float* __restrict__ lse,                         // lse of row 0 (stride 1) or null
    const KV& kv, int nq, int nk, int q0, int wg_rows, int r0, float scale, int causal,
    bf16_t* __restrict__ lds) {
  using L = PfLds<D>;
  static_assert(DEPTH == 1 || DEPTH == 2, "prefetch depth");
  constexpr int kThreads = 64 * W;
  constexpr int kCh = D / 8;                  // 16-byte chunks per row
  constexpr int kRowsPerIt = kThreads / kCh;
  constexpr int kIt = kPfBN / kRowsPerIt;     // K (and V) loads per thread per tile
  static_assert(kIt >= 1 && kPfBN % kRowsPerIt == 0, "tile staging layout");
  constexpr int kKs = D / 16;                 // MFMA k-steps over d
  constexpr int kDt = D / 32;                 // 32-row d tiles of O^T

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int l32 = lane & 31, half = lane >> 5;
  const int off = nk - nq;                    // bottom-right causal offset
  const int row = r0 + l32;

  const int wg_last = min(q0 + wg_rows, nq) - 1;
  const int kend = causal ? min(nk, wg_last + off + 1) : nk;
  const int w_last = min(r0 + 32, nq) - 1;
  const int kend_w = (r0 >= nq) ? 0 : (causal ? min(nk, w_last + off + 1) : nk);
  const int n_tiles = kend > 0 ? (kend + kPfBN - 1) / kPfBN : 0;

  // Q^T fragments (B operand): lane holds q[row][16*ks + 8*half .. +8].
  bf16x8 qf[kKs];
#pragma unroll
  for (int ks = 0; ks < kKs; ++ks) {
    u32x4 z = {0, 0, 0, 0};
    qf[ks] = as_bf16x8(row < nq ? load16(q + (size_t)row * q_stride + ks * 16 + half * 8) : z);
  }

  f32x16 oacc[kDt];
#pragma unroll
  for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) oacc[dt][j] = 0.f;

  const float c = scale * kLog2e;
  const float tau = kRescaleLog2 / c;
  float m_used = -INFINITY;
  float l = 0.f;

  // ---- staging: K and V rows copied as 16-byte chunks ----------------------
  // DEPTH register sets.  DEPTH 1: the loads of tile t+1 go out at the start
  // of step t and are written to LDS after its compute.  DEPTH 2: on entry to
  // step t the loads of tiles t+1 and t+2 are already in flight (one per set);
  // after the compute, tile t+1 is written to LDS and the loads of tile t+3 go
  // out into the set just freed, so every load has two steps to arrive.
  const int ld_ch = tid % kCh;
  const int ld_row = tid / kCh;
  struct Stage {
    u32x4 k[kIt], v[kIt];
  };
  Stage st0, st1;
  auto load_tile = [&](Stage& sg, int k0) {
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int j = k0 + it * kRowsPerIt + ld_row;
      u32x4 z = {0, 0, 0, 0};
      sg.k[it] = j < nk ? load16(kv.krow(j) + ld_ch * 8) : z;
      sg.v[it] = j < nk ? load16(kv.vrow(j) + ld_ch * 8) : z;
    }
  };
  auto store_tile = [&](const Stage& sg, int buf) {
    bf16_t* kl = lds + buf * L::kElemsBuf;
    bf16_t* vl = kl + L::kElemsK;
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int r = it * kRowsPerIt + ld_row;
      *reinterpret_cast<u32x4*>(kl + r * L::kStrK + ld_ch * 8) = sg.k[it];
      *reinterpret_cast<u32x4*>(vl + r * L::kStrV + ld_ch * 8) = sg.v[it];
    }
  };

  if (n_tiles > 0) {
    load_tile(st0, 0);
    if constexpr (DEPTH == 2) {
      if (n_tiles > 1) load_tile(st1, kPfBN);
      store_tile(st0, 0);
      if (n_tiles > 2) load_tile(st0, 2 * kPfBN);
    } else {
      store_tile(st0, 0);
    }
  }
  __syncthreads();

  // Transposing-read source address inside the V tile (see lds_read_tr4):
  // lane (group g = lane/16, r = lane%16) points at key 4*half + r/4 and
  // d = 16*(g%2) + 4*(r%4) of a 16-key slice; the group's result gives lane
  // l the values V[slice + 4*half + k][l%32], k = 0..3.
  const int g16 = lane >> 4, r16 = lane & 15;
  const int tr_off = (4 * half + (r16 >> 2)) * L::kStrV + 16 * (g16 & 1) + 4 * (r16 & 3);

  // Tile t is computed from LDS buffer t % 2; with DEPTH 2 the register set
  // holding tile t+1 is st1 for even t and st0 for odd t.
  auto step = [&](int t, Stage& cur) {
    const int k0 = t * kPfBN;
    if (DEPTH == 1 && t + 1 < n_tiles) load_tile(cur, k0 + kPfBN);
    const bf16_t* kl = lds + (t & 1) * L::kElemsBuf;
    const bf16_t* vl = kl + L::kElemsK;

    if (k0 < kend_w) {
      // ---- S^T = K Q^T for 64 keys x 32 rows -------------------------------
      // accumulator element j of m-tile mt holds key 32*mt + 8*(j/4) +
      // 4*half + j%4 of this lane's query row.
      f32x16 s[2];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int j = 0; j < 16; ++j) s[mt][j] = 0.f;
#pragma unroll
      for (int ks = 0; ks < kKs; ++ks) {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(
              kl + (32 * mt + l32) * L::kStrK + ks * 16 + half * 8);
          s[mt] = mfma32(a, qf[ks], s[mt]);
        }
      }
      // ---- mask (diagonal / ragged tiles only) -----------------------------
      const bool need_mask = (k0 + kPfBN > nk) || (causal && k0 + kPfBN - 1 > r0 + off);
      if (need_mask) {
        const int lim = causal ? min(nk - 1, row + off) : nk - 1;
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int key = k0 + 32 * mt + 8 * (j >> 2) + 4 * half + (j & 3);
            if (key > lim) s[mt][j] = -INFINITY;
          }
      }
      // ---- online softmax ----------------------------------------------------
      float tmax = s[0][0];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int j = 0; j < 16; ++j) tmax = fmaxf(tmax, s[mt][j]);
      tmax = fmaxf(tmax, wave_xor(tmax, 32));
      if (wave_any(tmax > m_used + tau)) {
        const float m_new = fmaxf(m_used, tmax);
        const float alpha = (m_used == -INFINITY) ? 0.f : fast_exp2((m_used - m_new) * c);
        l *= alpha;
#pragma unroll
        for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
          for (int j = 0; j < 16; ++j) oacc[dt][j] *= alpha;
        m_used = m_new;
      }
      const float mref = (m_used == -INFINITY) ? 0.f : m_used * c;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const float p = fast_exp2(fmaf(s[mt][j], c, -mref));
          s[mt][j] = p;
          l += p;
        }
      // ---- O^T += V^T P^T ----------------------------------------------------
      // k-step (mt, s2) covers keys 32*mt + 16*s2 + [0, 16); B-operand slot
      // 8*half + t is accumulator element 8*s2 + t, i.e. key
      // 32*mt + 16*s2 + 8*(t/4) + 4*half + t%4, which the two transposing
      // reads (slices +0 and +8) deliver in the same order.
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const int b = 8 * s2;
          const bf16x8 pb = to_bf16x8(s[mt][b], s[mt][b + 1], s[mt][b + 2], s[mt][b + 3],
                                      s[mt][b + 4], s[mt][b + 5], s[mt][b + 6], s[mt][b + 7]);
          const bf16_t* vs = vl + (32 * mt + 16 * s2) * L::kStrV + tr_off;
#pragma unroll
          for (int dt = 0; dt < kDt; ++dt) {
            const bf16x8 a = join_bf16x8(lds_read_tr4(vs + 32 * dt),
                                         lds_read_tr4(vs + 8 * L::kStrV + 32 * dt));
            oacc[dt] = mfma32(a, pb, oacc[dt]);
          }
        }
      }
    }
    if (t + 1 < n_tiles) store_tile(cur, (t + 1) & 1);
    if (DEPTH == 2 && t + 3 < n_tiles) load_tile(cur, k0 + 3 * kPfBN);
    __syncthreads();
  };
  int t = 0;
  for (; t + 1 < n_tiles; t += 2) {
    if constexpr (DEPTH == 2) {
      step(t, st1);
      step(t + 1, st0);
    } else {
      step(t, st0);
      step(t + 1, st0);
    }
  }
  if (t < n_tiles) step(t, DEPTH == 2 ? st1 : st0);

  // ---- epilogue: normalise, store bf16 rows and the log-sum-exp -------------
  const float lt = l + wave_xor(l, 32);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  if (row < nq) {
    bf16_t* orow = o + (size_t)row * o_stride;
#pragma unroll
    for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d = 32 * dt + 8 * g4 + 4 * half;
        const bf16x4 w = to_bf16x4(oacc[dt][4 * g4] * inv, oacc[dt][4 * g4 + 1] * inv,
                                   oacc[dt][4 * g4 + 2] * inv, oacc[dt][4 * g4 + 3] * inv);
        *reinterpret_cast<bf16x4*>(orow + d) = w;
      }
    if (lse != nullptr && half == 0)
      lse[row] = lt > 0.f ? m_used * scale + logf(lt) : -INFINITY;
  }
}

}  // namespace rag
