// Causal (or full) attention of one query tile against the keys of its
// sequence, for gfx950: W waves of 32 rows each, covering up to four q heads
// of one GQA group (which share every K/V tile) times the row blocks of the
// tile.
//
// Method: exact tiled attention with an online softmax (FlashAttention's
// forward pass; the running-max rescaling of Milakov & Gimelshein), laid out
// for CDNA4:
//   * each wave owns 32 query rows of one head and keeps them in registers as
//     the B operand of v_mfma_f32_32x32x16_bf16; K/V tiles of 64 keys are
//     shared through LDS by all waves (all heads of the group) of the tile;
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
//     end; tiles fully above the diagonal are skipped per wave;
//   * two ways to stage K/V: (a) DMA -- global_load_lds_dwordx4 writes the
//     tile straight into one of three LDS stages two tiles ahead of its use,
//     with XOR-swizzled rows so every LDS read group is conflict-free (dense
//     K/V); (b) registers -- 16-byte loads into registers, then LDS rows
//     padded against bank conflicts; this path can zero rows past the
//     sequence end, which a paged cache's tail slots need.
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

// ---------------------------------------------------------------------------
// LDS layouts of one K/V tile (64 keys, row-major [key][d]).  Each layout
// object holds the lane-dependent part of its read offsets, so that every
// LDS read in the tile loop is one register plus a compile-time immediate.
//   k_off(mt, ks): A-operand read of K rows 32*mt + l32, d = 16*ks + 8*half
//   v_off(r, dt):  transposing read of the V slice starting at row r (r a
//                  multiple of 8), d tile dt (see pf_tile)
// ---------------------------------------------------------------------------
// Padded rows (register staging): K rows +16 B, V rows +32 B (see PfLds).
template <int D>
struct PaddedLayout {
  using L = PfLds<D>;
  int k_lane, v_lane;
  __device__ __forceinline__ PaddedLayout() {
    const int lane = threadIdx.x & 63;
    const int l32 = lane & 31, half = lane >> 5, g16 = lane >> 4, r16 = lane & 15;
    k_lane = l32 * L::kStrK + 8 * half;
    v_lane = (4 * half + (r16 >> 2)) * L::kStrV + 16 * (g16 & 1) + 4 * (r16 & 3);
  }
  __device__ __forceinline__ int k_off(int mt, int ks) const {
    return 32 * mt * L::kStrK + 16 * ks + k_lane;
  }
  __device__ __forceinline__ int v_off(int r, int dt) const {
    return r * L::kStrV + 32 * dt + v_lane;
  }
};

// Unpadded rows with XOR-swizzled 16-byte chunks (DMA staging, whose lane
// order fixes 64 consecutive chunks per wave instruction).  K chunk c of row
// r sits at c ^ (r & 7): the eight rows an A-operand read group touches land
// in distinct banks.  V chunk c of row r sits at c ^ 2*(r & 3): the four rows
// x two chunks a transposing-read group touches land in distinct banks.
// Written out per lane, K offsets depend on the lane only through
// (ks & 3) ^ ((l32 >> 1) & 3) and V offsets through (dt & 1) ^ (r16 >> 3).
template <int D>
struct SwizzledLayout {
  static constexpr int kElemsTile = 2 * kPfBN * D;   // K then V
  int k_lane[4], v_lane[2];
  __device__ __forceinline__ SwizzledLayout() {
    const int lane = threadIdx.x & 63;
    const int l32 = lane & 31, half = lane >> 5, g16 = lane >> 4, r16 = lane & 15;
    const int x2 = (l32 >> 1) & 3, hh = half ^ (l32 & 1);
#pragma unroll
    for (int b = 0; b < 4; ++b) k_lane[b] = l32 * D + 16 * (b ^ x2) + 8 * hh;
    const int y = r16 >> 2;                                  // row & 3 of the source row
    const int cl = (2 * (g16 & 1) + ((r16 & 3) >> 1)) ^ (2 * (y & 1));
#pragma unroll
    for (int e = 0; e < 2; ++e)
      v_lane[e] = (4 * half + y) * D + 32 * (e ^ (y >> 1)) + 8 * cl + 4 * (r16 & 1);
  }
  __device__ __forceinline__ int k_off(int mt, int ks) const {
    return 32 * mt * D + 64 * (ks >> 2) + k_lane[ks & 3];
  }
  __device__ __forceinline__ int v_off(int r, int dt) const {
    return r * D + 64 * (dt >> 1) + v_lane[dt & 1];
  }
  // physical chunk of logical chunk c in row r (the DMA side)
  __device__ __forceinline__ static int k_phys(int r, int c) { return c ^ (r & 7); }
  __device__ __forceinline__ static int v_phys(int r, int c) { return c ^ (2 * (r & 3)); }
};

// ---------------------------------------------------------------------------
// Per-wave state and the per-tile compute shared by both staging paths.
// ---------------------------------------------------------------------------
template <int D>
struct PfState {
  bf16x8 qf[D / 16];    // Q^T fragments (B operand)
  f32x16 oacc[D / 32];  // O^T accumulators (32-row d tiles)
  float m_used, l;
};

template <int D>
__device__ __forceinline__ void pf_init(PfState<D>& st, const bf16_t* __restrict__ q,
                                        size_t q_stride, int row, int nq) {
  const int half = (threadIdx.x & 63) >> 5;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    u32x4 z = {0, 0, 0, 0};
    st.qf[ks] =
        as_bf16x8(row < nq ? load16(q + (size_t)row * q_stride + ks * 16 + half * 8) : z);
  }
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) st.oacc[dt][j] = 0.f;
  st.m_used = -INFINITY;
  st.l = 0.f;
}

// One 64-key tile for this wave's 32 rows [r0, r0 + 32).
template <int D, class Layout>
__device__ __forceinline__ void pf_tile(PfState<D>& st, const Layout& lay,
                                        const bf16_t* __restrict__ kl,
                                        const bf16_t* __restrict__ vl, int k0, int r0, int nk,
                                        int off, int causal, float c, float tau) {
  constexpr int kKs = D / 16;
  constexpr int kDt = D / 32;
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31, half = lane >> 5;
  const int row = r0 + l32;

  // ---- S^T = K Q^T for 64 keys x 32 rows ------------------------------------
  // accumulator element j of m-tile mt holds key 32*mt + 8*(j/4) + 4*half +
  // j%4 of this lane's query row.
  f32x16 s[2];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int j = 0; j < 16; ++j) s[mt][j] = 0.f;
#pragma unroll
  for (int ks = 0; ks < kKs; ++ks) {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(kl + lay.k_off(mt, ks));
      s[mt] = mfma32(a, st.qf[ks], s[mt]);
    }
  }
  // ---- mask (diagonal / ragged tiles only) ----------------------------------
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
  // ---- online softmax ---------------------------------------------------------
  float tmax = s[0][0];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int j = 0; j < 16; ++j) tmax = fmaxf(tmax, s[mt][j]);
  tmax = fmaxf(tmax, wave_xor(tmax, 32));
  if (wave_any(tmax > st.m_used + tau)) {
    const float m_new = fmaxf(st.m_used, tmax);
    const float alpha = (st.m_used == -INFINITY) ? 0.f : fast_exp2((st.m_used - m_new) * c);
    st.l *= alpha;
#pragma unroll
    for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
      for (int j = 0; j < 16; ++j) st.oacc[dt][j] *= alpha;
    st.m_used = m_new;
  }
  const float mref = (st.m_used == -INFINITY) ? 0.f : st.m_used * c;
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float p = fast_exp2(fmaf(s[mt][j], c, -mref));
      s[mt][j] = p;
      st.l += p;
    }
  // ---- O^T += V^T P^T ---------------------------------------------------------
  // k-step (mt, s2) covers keys 32*mt + 16*s2 + [0, 16); B-operand slot
  // 8*half + t is accumulator element 8*s2 + t, i.e. key
  // 32*mt + 16*s2 + 8*(t/4) + 4*half + t%4, which the two transposing reads
  // (slices +0 and +8) deliver in the same order.  Transposing-read source:
  // lane (group g = lane/16, r = lane%16) points at key slice + 4*half + r/4,
  // d = 32*dt + 16*(g%2) + 4*(r%4); the group's result gives lane l the
  // values V[slice + 4*half + k][32*dt + l%32], k = 0..3.
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const int b = 8 * s2;
      const bf16x8 pb = to_bf16x8(s[mt][b], s[mt][b + 1], s[mt][b + 2], s[mt][b + 3],
                                  s[mt][b + 4], s[mt][b + 5], s[mt][b + 6], s[mt][b + 7]);
      const int rw = 32 * mt + 16 * s2;
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt) {
        const bf16x8 a = join_bf16x8(lds_read_tr4(vl + lay.v_off(rw, dt)),
                                     lds_read_tr4(vl + lay.v_off(rw + 8, dt)));
        st.oacc[dt] = mfma32(a, pb, st.oacc[dt]);
      }
    }
  }
}

// Normalise and store this wave's rows and their log-sum-exp.
template <int D>
__device__ __forceinline__ void pf_store(const PfState<D>& st, bf16_t* __restrict__ o,
                                         size_t o_stride, float* __restrict__ lse, int row,
                                         int nq, float scale) {
  const int half = (threadIdx.x & 63) >> 5;
  const float lt = st.l + wave_xor(st.l, 32);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  if (row >= nq) return;
  bf16_t* orow = o + (size_t)row * o_stride;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int d = 32 * dt + 8 * g4 + 4 * half;
      const bf16x4 w = to_bf16x4(st.oacc[dt][4 * g4] * inv, st.oacc[dt][4 * g4 + 1] * inv,
                                 st.oacc[dt][4 * g4 + 2] * inv, st.oacc[dt][4 * g4 + 3] * inv);
      *reinterpret_cast<bf16x4*>(orow + d) = w;
    }
  if (lse != nullptr && half == 0)
    lse[row] = lt > 0.f ? st.m_used * scale + logf(lt) : -INFINITY;
}

// Key range of the workgroup and of this wave.
struct PfRange {
  int off, n_tiles, kend_w;
};
__device__ __forceinline__ PfRange pf_range(int nq, int nk, int q0, int wg_rows, int r0,
                                            int causal) {
  PfRange r;
  r.off = nk - nq;                              // bottom-right causal offset
  const int wg_last = min(q0 + wg_rows, nq) - 1;
  const int kend = causal ? min(nk, wg_last + r.off + 1) : nk;
  const int w_last = min(r0 + 32, nq) - 1;
  r.kend_w = (r0 >= nq) ? 0 : (causal ? min(nk, w_last + r.off + 1) : nk);
  r.n_tiles = kend > 0 ? (kend + kPfBN - 1) / kPfBN : 0;
  return r;
}

// ---------------------------------------------------------------------------
// Register-staged tile loop (padded LDS rows, double buffer, one tile ahead).
// q, o and lse point at row 0 of the sequence for this wave's head; the
// workgroup (W waves) covers rows [q0, q0 + wg_rows) and this wave rows
// [r0, r0 + 32).  Rows past the sequence end are staged as zeros.
// ---------------------------------------------------------------------------
template <int D, int W, class KV>
__device__ __forceinline__ void prefill_tile_regs(
    const bf16_t* __restrict__ q, size_t q_stride, bf16_t* __restrict__ o, size_t o_stride,
    float* __restrict__ lse, const KV& kv, int nq, int nk, int q0, int wg_rows, int r0,
    float scale, int causal, bf16_t* __restrict__ lds) {
  using L = PfLds<D>;
  constexpr int kThreads = 64 * W;
  constexpr int kCh = D / 8;                  // 16-byte chunks per row
  constexpr int kRowsPerIt = kThreads / kCh;
  constexpr int kIt = kPfBN / kRowsPerIt;     // K (and V) loads per thread per tile
  static_assert(kIt >= 1 && kPfBN % kRowsPerIt == 0, "tile staging layout");
  const int tid = threadIdx.x;
  const PfRange rg = pf_range(nq, nk, q0, wg_rows, r0, causal);
  const float c = scale * kLog2e;
  const float tau = kRescaleLog2 / c;

  PfState<D> st;
  pf_init(st, q, q_stride, r0 + (tid & 31), nq);

  const int ld_ch = tid % kCh;
  const int ld_row = tid / kCh;
  u32x4 kreg[kIt], vreg[kIt];
  auto load_tile = [&](int k0) {
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int j = k0 + it * kRowsPerIt + ld_row;
      u32x4 z = {0, 0, 0, 0};
      kreg[it] = j < nk ? load16(kv.krow(j) + ld_ch * 8) : z;
      vreg[it] = j < nk ? load16(kv.vrow(j) + ld_ch * 8) : z;
    }
  };
  auto store_tile = [&](int buf) {
    bf16_t* kl = lds + buf * L::kElemsBuf;
    bf16_t* vl = kl + L::kElemsK;
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int r = it * kRowsPerIt + ld_row;
      *reinterpret_cast<u32x4*>(kl + r * L::kStrK + ld_ch * 8) = kreg[it];
      *reinterpret_cast<u32x4*>(vl + r * L::kStrV + ld_ch * 8) = vreg[it];
    }
  };

  const PaddedLayout<D> lay;
  if (rg.n_tiles > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();
  for (int t = 0; t < rg.n_tiles; ++t) {
    const int k0 = t * kPfBN;
    if (t + 1 < rg.n_tiles) load_tile(k0 + kPfBN);
    const bf16_t* kl = lds + (t & 1) * L::kElemsBuf;
    if (k0 < rg.kend_w)
      pf_tile<D>(st, lay, kl, kl + L::kElemsK, k0, r0, nk, rg.off, causal, c, tau);
    if (t + 1 < rg.n_tiles) store_tile((t + 1) & 1);
    __syncthreads();
  }
  pf_store(st, o, o_stride, lse, r0 + (tid & 31), nq, scale);
}

// ---------------------------------------------------------------------------
// DMA-staged tile loop for dense K/V (three LDS stages s0/s1/s2 of
// SwizzledLayout).  The loads of tile t+2 go out at the start of step t into
// the stage tile t-1 used; at the end of step t the wave waits until its
// loads of tile t+1 have landed, then the workgroup barrier makes every
// wave's share visible.  Rows past the sequence end are loaded from its last
// row (finite data; those keys are masked).
// ---------------------------------------------------------------------------
template <int D, int W>
__device__ __forceinline__ void prefill_tile_dma(
    const bf16_t* __restrict__ q, size_t q_stride, bf16_t* __restrict__ o, size_t o_stride,
    float* __restrict__ lse, const DenseKV& kv, int nq, int nk, int q0, int wg_rows, int r0,
    float scale, int causal, bf16_t* __restrict__ s0, bf16_t* __restrict__ s1,
    bf16_t* __restrict__ s2) {
  using Lay = SwizzledLayout<D>;
  constexpr int kCh = D / 8;                     // 16-byte chunks per row
  constexpr int kInstr = kPfBN * kCh / (64 * W);  // K (and V) DMA instructions per wave per tile
  static_assert(kInstr >= 1 && (kPfBN * kCh) % (64 * W) == 0, "tile staging layout");
  constexpr int kLoadsPerTile = 2 * kInstr;      // vmcnt events per wave per tile
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const PfRange rg = pf_range(nq, nk, q0, wg_rows, r0, causal);
  const float c = scale * kLog2e;
  const float tau = kRescaleLog2 / c;

  PfState<D> st;
  pf_init(st, q, q_stride, r0 + (lane & 31), nq);

  // Instruction i of this wave writes physical chunks [64*gi, 64*gi + 64) of
  // the tile, gi = wave*kInstr + i; lane l's chunk P = 64*gi + l is physical
  // chunk P % kCh of row P / kCh, which holds logical chunk phys ^ swizzle.
  auto issue_tile = [&](bf16_t* stage, int k0) {
    typedef __attribute__((address_space(3))) void lds_void;
#pragma unroll
    for (int i = 0; i < kInstr; ++i) {
      const int gi = wave * kInstr + i;
      const int p = 64 * gi + lane;
      const int r = p / kCh, phys = p % kCh;
      const int j = min(k0 + r, nk - 1);
      const bf16_t* ksrc = kv.krow(j) + Lay::k_phys(r, phys) * 8;
      const bf16_t* vsrc = kv.vrow(j) + Lay::v_phys(r, phys) * 8;
      __builtin_amdgcn_global_load_lds(ksrc, (lds_void*)(stage + 64 * gi * 8), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(vsrc, (lds_void*)(stage + kPfBN * D + 64 * gi * 8), 16,
                                       0, 0);
    }
  };
  // vmcnt(n): wait until at most n vector-memory operations of this wave are
  // outstanding (gfx9 encoding: vmcnt in bits 3:0 and 15:14; expcnt and
  // lgkmcnt left at their maximum, i.e. not waited on).
  auto wait_vm = [](bool keep_one_tile) {
    if (keep_one_tile)
      __builtin_amdgcn_s_waitcnt(0x0F70 | (kLoadsPerTile & 15) | ((kLoadsPerTile >> 4) << 14));
    else
      __builtin_amdgcn_s_waitcnt(0x0F70);
  };

  const Lay lay;
  const int nt = rg.n_tiles;
  if (nt > 0) issue_tile(s0, 0);
  if (nt > 1) issue_tile(s1, kPfBN);
  wait_vm(nt > 1);
  __builtin_amdgcn_s_barrier();

  auto step = [&](int t, const bf16_t* cur, bf16_t* ahead) {
    const int k0 = t * kPfBN;
    if (t + 2 < nt) issue_tile(ahead, k0 + 2 * kPfBN);
    if (k0 < rg.kend_w)
      pf_tile<D>(st, lay, cur, cur + kPfBN * D, k0, r0, nk, rg.off, causal, c, tau);
    wait_vm(t + 2 < nt);
    __builtin_amdgcn_s_barrier();
  };
  int t = 0;
  for (; t + 2 < nt; t += 3) {
    step(t, s0, s2);
    step(t + 1, s1, s0);
    step(t + 2, s2, s1);
  }
  if (t < nt) step(t, s0, s2);
  if (t + 1 < nt) step(t + 1, s1, s0);
  pf_store(st, o, o_stride, lse, r0 + (lane & 31), nq, scale);
}

}  // namespace rag
