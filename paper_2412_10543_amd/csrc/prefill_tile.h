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
// Padded rows (register staging): K rows +16 B, V rows +64 B (see PfLds).
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

// DMA staging layout.  A DMA instruction writes 64 consecutive 16-byte
// chunks (lane l at +16*l) but may gather them from anywhere, so the tile is
// stored chunk-permuted.  gfx950's LDS has 64 four-byte banks; a 16-byte read
// is serviced 16 lanes at a time and an 8-byte (transposing) read 32 lanes at
// a time, and each such group must touch every bank once.
//   K: chunk c of row r at chunk (r/16)*16*kCh + 16*c + r%16 -- the 16 rows
//      of an A-operand read group are 16 consecutive chunks;
//   V: the 32-d tiles (four chunks of a row) are stored one after another,
//      each 64 rows x 64 bytes row-major -- the 4 rows x 64 bytes of a
//      transposing read group are 256 consecutive bytes.
// Every read is then one per-lane register (k_lane or v_lane) plus a
// compile-time offset, and no read group hits a bank twice.
template <int D>
struct ChunkLayout {
  static constexpr int kCh = D / 8;                  // 16-byte chunks per row
  static constexpr int kElemsTile = 2 * kPfBN * D;   // K then V
  int k_lane, v_lane;                                // in bf16 elements
  __device__ __forceinline__ ChunkLayout() {
    const int lane = threadIdx.x & 63;
    const int l32 = lane & 31, half = lane >> 5, g16 = lane >> 4, r16 = lane & 15;
    // K read: row 32*mt + l32, chunk 2*ks + half
    k_lane = (l32 >> 4) * 128 * kCh + 128 * half + 8 * (l32 & 15);
    // V read: row slice + 4*half + r16/4, bytes 64*dt + 32*(g16 % 2) + 8*(r16 % 4)
    v_lane = 32 * (4 * half + (r16 >> 2)) + 16 * (g16 & 1) + 4 * (r16 & 3);
  }
  __device__ __forceinline__ int k_off(int mt, int ks) const {
    return k_lane + 256 * kCh * mt + 256 * ks;
  }
  __device__ __forceinline__ int v_off(int r, int dt) const {
    return v_lane + 2048 * dt + 32 * r;
  }
  // (row, chunk) of the tile held by staged chunk p (the DMA side)
  __device__ __forceinline__ static void k_src(int p, int& r, int& c) {
    r = (p / (16 * kCh)) * 16 + (p & 15);
    c = (p >> 4) % kCh;
  }
  __device__ __forceinline__ static void v_src(int p, int& r, int& c) {
    r = (p & 255) >> 2;
    c = 4 * (p >> 8) + (p & 3);
  }
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
// Software-pipelined tile loop for dense K/V (DMA staging into four LDS
// stages of ChunkLayout).
//
// The unit of work is a block of 32 keys (half a tile).  For block b a wave
// does QK(b) (S^T of 32 keys x its 32 rows: D/16 MFMAs), SM(b) (exp2 of the
// scores, bf16 packing, row sums: vector ALU) and PV(b) (D/16 MFMAs).  Slot b
// issues QK(b+1) and PV(b-1) on the matrix cores while SM(b) runs on the
// vector ALU, so within each wave the two units work side by side instead of
// taking turns (the two waves sharing a SIMD are held in step by the
// per-tile barrier, so they could not fill each other's gaps).
//
// Each block is one online-softmax step.  Its weights are formed against the
// current exponent reference m (the running maximum as last moved) and kept
// if every lane's sum of its 16 weights is at most kPfSumBound, which bounds
// each weight; otherwise -- the first block of a row (m = -inf makes the sum
// inf or NaN), or scores far above m -- the block is redone exactly: m moves
// to the new row maximum, output and sum are rescaled, weights recomputed.
//
// Stages: tile t lives in stage t % 4.  Slot 2t reads K of tile t (keys
// 32..63) and V of tile t-1 (keys 32..63); slot 2t+1 reads K of tile t+1
// (keys 0..31) and V of tile t (keys 0..31).  Between the two slots each wave
// waits for its share of tile t+1, the workgroup barrier publishes it and
// retires tile t-1, and the DMA of tile t+3 goes out into tile t-1's stage.
// ---------------------------------------------------------------------------
constexpr float kPfSumBound = 65536.f;   // 2^16: weights stay far inside fp32/bf16 range

// Max of x over the two 32-lane halves (lanes l and l ^ 32 hold one row).
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                  false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Workgroup barrier that no LDS access is moved across, by the compiler's IR
// passes or by its instruction scheduler.
__device__ __forceinline__ void pf_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// S^T of the 32 keys [32*H, 32*H + 32) of a staged tile against this wave's
// rows; element j of the result is key 8*(j/4) + 4*half + j%4 of the block.
template <int D, int H>
__device__ __forceinline__ f32x16 pf_qk(const PfState<D>& st, const ChunkLayout<D>& lay,
                                        const bf16_t* __restrict__ kst) {
  f32x16 s = {};
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const bf16x8 a = *reinterpret_cast<const bf16x8*>(kst + lay.k_off(H, ks));
    s = mfma32(a, st.qf[ks], s);
  }
  return s;
}

// O^T += V^T P^T over the keys [32*H, 32*H + 32) of a staged tile (stage =
// the tile's K then V); p[s2] is
// the B operand of keys 16*s2 .. +16 of the block (see pf_tile for the order).
template <int D, int H>
__device__ __forceinline__ void pf_pv(PfState<D>& st, const ChunkLayout<D>& lay,
                                      const bf16_t* __restrict__ stage, const bf16x8 (&p)[2]) {
  const bf16_t* vst = stage + kPfBN * D;   // V follows K in a stage
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2) {
    const int rw = 32 * H + 16 * s2;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
      const bf16x8 a = join_bf16x8(lds_read_tr4(vst + lay.v_off(rw, dt)),
                                   lds_read_tr4(vst + lay.v_off(rw + 8, dt)));
      st.oacc[dt] = mfma32(a, p[s2], st.oacc[dt]);
    }
  }
}

// Weights 2^(s*c + nm) of one block, packed to bf16 in pf_pv's operand order;
// returns this lane's fp32 sum of the weights.
__device__ __forceinline__ float pf_weights(const f32x16& s, float c, float nm,
                                            bf16x8 (&p)[2]) {
  float w[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) w[j] = fast_exp2(fmaf(s[j], c, nm));
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < 16; ++j) sum += w[j];
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2) {
    const int b = 8 * s2;
    p[s2] = to_bf16x8(w[b], w[b + 1], w[b + 2], w[b + 3], w[b + 4], w[b + 5], w[b + 6],
                      w[b + 7]);
  }
  return sum;
}

// Keys past lim (this lane's last visible key) of the block starting at key0.
__device__ __forceinline__ void pf_mask(f32x16& s, int key0, int lim) {
  const int half = (threadIdx.x & 63) >> 5;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int key = key0 + 8 * (j >> 2) + 4 * half + (j & 3);
    if (key > lim) s[j] = -INFINITY;
  }
}

// The exact path: move m to the row maximum, rescale, recompute the weights.
template <int D>
__device__ __forceinline__ float pf_reref(PfState<D>& st, const f32x16& s, float c,
                                          bf16x8 (&p)[2]) {
  // A side effect keeps the compiler from executing this rare path
  // unconditionally and selecting its results.
  asm volatile("");
  float tmax = s[0];
#pragma unroll
  for (int j = 1; j < 16; ++j) tmax = fmaxf(tmax, s[j]);
  tmax = max_halves(tmax);
  const float m_new = fmaxf(st.m_used, tmax);
  const float alpha = (st.m_used == -INFINITY) ? 0.f : fast_exp2((st.m_used - m_new) * c);
  st.l *= alpha;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) st.oacc[dt][j] *= alpha;
  st.m_used = m_new;
  return pf_weights(s, c, (m_new == -INFINITY) ? 0.f : -m_new * c, p);
}

// Per-wave constants of the pipelined loop.
struct PfPipeCtx {
  float c;     // scale * log2(e)
  int nbw;     // 32-key blocks this wave computes
  int lim;     // last key this lane's row sees
  int mlim;    // blocks ending past this key need masking
};

// A full slot in an explicit instruction order: D/16 steps, each with the
// LDS operand reads of the step two ahead, one QK(b+1) MFMA, vector work of
// SM(b), one PV(b-1) MFMA.  The vector work is itself pipelined over the
// steps -- step i forms the exponent arguments of step i+1's scores, the
// exponentials of step i's and packs and sums step i-1's -- so no vector
// instruction waits on the one before it (a wave issues in order, and such
// a wait would hold back its next MFMA too).  A scheduling barrier after each
// step and empty asm statements on the values each step produces keep the
// compiler from regrouping the work (left alone it clusters the MFMAs, and
// the two units take turns).
template <int D, int HK, int HV>
__device__ __forceinline__ float pf_full_slot(PfState<D>& st, const ChunkLayout<D>& lay,
                                              const bf16_t* __restrict__ kst,
                                              const bf16_t* __restrict__ vstage,
                                              const f32x16& s_cur, f32x16& s_next,
                                              bf16x8 (&p_cur)[2], const bf16x8 (&p_prev)[2],
                                              float c, float nm) {
  const bf16_t* vst = vstage + kPfBN * D;   // V follows K in a stage
  constexpr int kSteps = D / 16;          // QK MFMAs = PV MFMAs = steps
  constexpr int kDt = D / 32;
  constexpr int kPer = 16 / kSteps;       // scores (per lane) per step
  static_assert(kPer % 2 == 0 && 16 % kSteps == 0, "step shape");
  bf16x8 ka[kSteps], va[kSteps];
  auto load = [&](int i) {
    ka[i] = *reinterpret_cast<const bf16x8*>(kst + lay.k_off(HK, i));
    const int rw = 32 * HV + 16 * (i / kDt), dt = i % kDt;
    va[i] = join_bf16x8(lds_read_tr4(vst + lay.v_off(rw, dt)),
                        lds_read_tr4(vst + lay.v_off(rw + 8, dt)));
  };
  float x[16], w[16];
  bf16x2 pr[8];
  float sum = 0.f;
  auto arg = [&](int i) {          // exponent arguments of step i's scores
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      x[i * kPer + u] = fmaf(s_cur[i * kPer + u], c, nm);
      asm volatile("" : "+v"(x[i * kPer + u]));
    }
  };
  auto expo = [&](int i) {
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      w[i * kPer + u] = fast_exp2(x[i * kPer + u]);
      asm volatile("" : "+v"(w[i * kPer + u]));
    }
  };
  auto pack = [&](int i) {         // bf16 pairs and the row sum
#pragma unroll
    for (int u = 0; u < kPer; u += 2) {
      const int e = i * kPer + u;
      f32x2 pw = {w[e], w[e + 1]};
      pr[e / 2] = __builtin_convertvector(pw, bf16x2);
      asm volatile("" : "+v"(pr[e / 2]));
      sum += w[e];
      sum += w[e + 1];
    }
    asm volatile("" : "+v"(sum));
  };
  load(0);
  if (kSteps > 1) load(1);
  arg(0);
  f32x16 acc = {};
#pragma unroll
  for (int i = 0; i < kSteps; ++i) {
    if (i + 2 < kSteps) load(i + 2);
    __builtin_amdgcn_sched_barrier(0);
    acc = mfma32(ka[i], st.qf[i], acc);
    if (i + 1 < kSteps) arg(i + 1);
    expo(i);
    if (i >= 1) pack(i - 1);
    st.oacc[i % kDt] = mfma32(va[i], p_prev[i / kDt], st.oacc[i % kDt]);
    __builtin_amdgcn_sched_barrier(0);
  }
  pack(kSteps - 1);
  s_next = acc;
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2)
    p_cur[s2] = __builtin_shufflevector(
        __builtin_shufflevector(pr[4 * s2], pr[4 * s2 + 1], 0, 1, 2, 3),
        __builtin_shufflevector(pr[4 * s2 + 2], pr[4 * s2 + 3], 0, 1, 2, 3), 0, 1, 2, 3, 4,
        5, 6, 7);
  return sum;
}

// Slot b: SM(b) on s_cur -> p_cur; QK(b+1) -> s_next from keys 32*HK.. of
// the stage kst; PV(b-1) with p_prev over keys 32*HV.. of the stage vst.
template <int D, int HK, int HV>
__device__ __forceinline__ void pf_slot(PfState<D>& st, const ChunkLayout<D>& lay,
                                        const PfPipeCtx& cx, int b, f32x16& s_cur,
                                        f32x16& s_next, bf16x8 (&p_cur)[2],
                                        const bf16x8 (&p_prev)[2], const bf16_t* kst,
                                        const bf16_t* vst) {
  const bool do_sm = b < cx.nbw;
  const bool do_qk = b + 1 < cx.nbw;
  const bool do_pv = b >= 1 && b <= cx.nbw;
  if (do_sm && 32 * b + 31 > cx.mlim) pf_mask(s_cur, 32 * b, cx.lim);
  if (do_sm && do_qk && do_pv) {
    float sum = pf_full_slot<D, HK, HV>(st, lay, kst, vst, s_cur, s_next, p_cur, p_prev, cx.c,
                                        -st.m_used * cx.c);
    if (__builtin_expect(wave_any(!(sum <= kPfSumBound)), 0))
      sum = pf_reref(st, s_cur, cx.c, p_cur);
    st.l += sum;
    return;
  }
  if (do_qk) s_next = pf_qk<D, HK>(st, lay, kst);
  if (do_pv) pf_pv<D, HV>(st, lay, vst, p_prev);
  if (do_sm) {
    float sum = pf_weights(s_cur, cx.c, -st.m_used * cx.c, p_cur);
    if (__builtin_expect(wave_any(!(sum <= kPfSumBound)), 0))
      sum = pf_reref(st, s_cur, cx.c, p_cur);
    st.l += sum;
  }
}

template <int D, int W>
__device__ __forceinline__ void prefill_tile_pipe(
    const bf16_t* __restrict__ q, size_t q_stride, bf16_t* __restrict__ o, size_t o_stride,
    float* __restrict__ lse, const DenseKV& kv, int nq, int nk, int q0, int wg_rows, int r0,
    float scale, int causal, bf16_t* __restrict__ s0, bf16_t* __restrict__ s1,
    bf16_t* __restrict__ s2, bf16_t* __restrict__ s3) {
  using Lay = ChunkLayout<D>;
  constexpr int kCh = D / 8;                     // 16-byte chunks per row
  constexpr int kInstr = kPfBN * kCh / (64 * W);  // K (and V) DMA instructions per wave per tile
  static_assert(kInstr >= 1 && (kPfBN * kCh) % (64 * W) == 0, "tile staging layout");
  constexpr int kLoadsPerTile = 2 * kInstr;      // vmcnt events per wave per tile
  static_assert(2 * kLoadsPerTile < 64, "vmcnt range");
  const int tid = threadIdx.x;
  const int wave = wave_id(), lane = tid & 63;
  const PfRange rg = pf_range(nq, nk, q0, wg_rows, r0, causal);
  const int row = r0 + (lane & 31);
  PfPipeCtx cx;
  cx.c = scale * kLog2e;
  cx.nbw = (rg.kend_w + 31) >> 5;
  cx.lim = causal ? min(nk - 1, row + rg.off) : nk - 1;
  cx.mlim = causal ? min(nk - 1, r0 + rg.off) : nk - 1;

  PfState<D> st;
  pf_init(st, q, q_stride, row, nq);

  // Instruction i of this wave writes staged chunks [64*gi, 64*gi + 64) of
  // the K and of the V region, gi = wave*kInstr + i; lane l fetches the
  // (row, chunk) that staged chunk 64*gi + l holds.  Rows past the sequence
  // end are loaded from its last row (finite data; those keys are masked).
  auto issue_tile = [&](bf16_t* stage, int k0) {
#pragma unroll
    for (int i = 0; i < kInstr; ++i) {
      const int gi = wave * kInstr + i;
      const int p = 64 * gi + lane;
      int kr, kc, vr, vc;
      Lay::k_src(p, kr, kc);
      Lay::v_src(p, vr, vc);
      dma16(kv.krow(min(k0 + kr, nk - 1)) + kc * 8, stage + 64 * gi * 8);
      dma16(kv.vrow(min(k0 + vr, nk - 1)) + vc * 8, stage + kPfBN * D + 64 * gi * 8);
    }
  };
  // Wait until at most `tiles` tiles of this wave's DMA are in flight
  // (vmcnt in bits 3:0 and 15:14; expcnt and lgkmcnt left at their maximum).
  auto wait_tiles = [](int tiles) {
    constexpr int k1 = kLoadsPerTile, k2 = 2 * kLoadsPerTile;
    if (tiles >= 2)
      __builtin_amdgcn_s_waitcnt(0x0F70 | (k2 & 15) | ((k2 >> 4) << 14));
    else if (tiles == 1)
      __builtin_amdgcn_s_waitcnt(0x0F70 | (k1 & 15) | ((k1 >> 4) << 14));
    else
      __builtin_amdgcn_s_waitcnt(0x0F70);
  };

  const Lay lay;
  const int nt = rg.n_tiles;
  if (nt > 0) issue_tile(s0, 0);
  // Take delivery of Q here (with tile 0, both needed first): the compiler
  // does not see the DMA, so a first use of Q inside the loop would make it
  // wait there for every copy in flight, on every iteration.
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) asm volatile("" : "+v"(st.qf[ks]));
  if (nt > 1) issue_tile(s1, kPfBN);
  if (nt > 2) issue_tile(s2, 2 * kPfBN);
  wait_tiles(min(nt, 3) - 1);
  pf_barrier();

  f32x16 sE = {}, sO = {};
  bf16x8 pE[2] = {}, pO[2] = {};
  if (cx.nbw > 0) sE = pf_qk<D, 0>(st, lay, s0);

  // Stage roles rotate by one each tile (tile t is in stage t % 4): prev
  // holds tile t-1 and, once the barrier has retired it, receives tile t+3.
  bf16_t* prev = s3;
  bf16_t* cur = s0;
  bf16_t* next = s1;
  bf16_t* after = s2;
  auto rotate = [&]() {
    bf16_t* const retired = prev;
    prev = cur;
    cur = next;
    next = after;
    after = retired;
  };
  // Any tile: slots decide per block what to do (first and last blocks,
  // masks, DMA near the end).
  auto general_step = [&](int t) {
    pf_slot<D, 1, 1>(st, lay, cx, 2 * t, sE, sO, pE, pO, cur, prev);
    wait_tiles(t + 2 < nt ? 1 : 0);
    pf_barrier();
    if (t + 3 < nt) issue_tile(prev, (t + 3) * kPfBN);
    pf_slot<D, 0, 0>(st, lay, cx, 2 * t + 1, sO, sE, pO, pE, next, cur);
  };
  // A tile whose two slots are full and unmasked for every wave and whose
  // DMA is due: straight-line code (a separate loop, so that its values never
  // meet the general path's at a join, which would cost register copies).
  auto steady_step = [&](int t) {
    float sum = pf_full_slot<D, 1, 1>(st, lay, cur, prev, sE, sO, pE, pO, cx.c,
                                      -st.m_used * cx.c);
    if (__builtin_expect(wave_any(!(sum <= kPfSumBound)), 0)) sum = pf_reref(st, sE, cx.c, pE);
    st.l += sum;
    wait_tiles(1);
    pf_barrier();
    issue_tile(prev, (t + 3) * kPfBN);
    sum = pf_full_slot<D, 0, 0>(st, lay, next, cur, sO, sE, pO, pE, cx.c, -st.m_used * cx.c);
    if (__builtin_expect(wave_any(!(sum <= kPfSumBound)), 0)) sum = pf_reref(st, sO, cx.c, pO);
    st.l += sum;
  };
  // Steady tiles are [1, t_end): the workgroup's first row block has the
  // fewest visible keys, so its limits bind every wave.  Tile t needs blocks
  // up to 2t+2 computed (2t+2 < nbw), keys up to 64t+63 unmasked and the DMA
  // of tile t+3 to exist.
  int t_end;
  {
    const int kend0 = causal ? min(nk, min(q0 + 32, nq) + rg.off) : nk;
    const int nbw0 = q0 >= nq ? 0 : (kend0 + 31) >> 5;
    const int mlim0 = causal ? min(nk - 1, q0 + rg.off) : nk - 1;
    const int a = nbw0 >= 3 ? (nbw0 - 3) / 2 + 1 : 0;
    const int b = mlim0 >= 63 ? (mlim0 - 63) / 64 + 1 : 0;
    t_end = min(min(a, b), nt - 3);
  }
  int t = 0;
  for (; t < min(nt, 1); ++t) {
    general_step(t);
    rotate();
  }
  for (; t < t_end; ++t) {
    steady_step(t);
    rotate();
  }
  for (; t < nt; ++t) {
    general_step(t);
    rotate();
  }
  // PV of the last block, when this wave computes the whole last tile (its
  // stage is now prev).
  if (nt > 0 && cx.nbw == 2 * nt) pf_pv<D, 1>(st, lay, prev, pO);
  pf_store(st, o, o_stride, lse, row, nq, scale);
}

}  // namespace rag
