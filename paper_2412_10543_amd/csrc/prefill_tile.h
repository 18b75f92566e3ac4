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
//     needs them; the matching V^T A operand comes straight from the V tile
//     through the transposing LDS read (ds_read_b64_tr_b16), so no data is
//     shuffled between the two products;
//   * K/V tiles go from HBM straight into LDS (global_load_lds_dwordx4),
//     four stages, issued three tiles ahead; dense rows or pages of a paged
//     cache (each DMA instruction covers one page);
//   * the work of each wave is software-pipelined over blocks of 32 keys so
//     that the matrix cores and the vector ALU work side by side;
//   * softmax statistics in fp32 with exp2 and the scale folded into one
//     FMA; the exponent reference moves only when a block's weights would
//     grow past 2^16, which keeps rescales of the output off the common path;
//   * masking only on blocks that cross the causal diagonal or the sequence
//     end; blocks fully above the diagonal are skipped per wave.
#pragma once

#include "common.h"

namespace rag {

// K/V rows of one (sequence, kv head) stored densely: token j at k + j*stride.
struct DenseKV {
  static constexpr bool kPaged = false;
  const bf16_t* k;
  const bf16_t* v;
  size_t stride;
  __device__ __forceinline__ const bf16_t* krow(int j) const { return k + (size_t)j * stride; }
  __device__ __forceinline__ const bf16_t* vrow(int j) const { return v + (size_t)j * stride; }
};

// K/V rows of one (sequence, kv head) in a paged cache: token j lives in
// physical block table[j / 16], slot j % 16.  k and v point at the kv head
// inside block 0; block_stride is the distance between blocks.  A DMA
// instruction covers 16 consecutive rows of a tile, i.e. one page, so its
// page id is the same for the whole wave and is read with a scalar load.
template <int D>
struct PagedDmaKV {
  static constexpr bool kPaged = true;
  const bf16_t* k;
  const bf16_t* v;
  const int32_t* table;
  size_t block_stride;
  // The block table is read-only for the whole launch; reading it through
  // the constant address space lets the wave-uniform reads be scalar loads
  // (a vector load would make the compiler wait for every DMA in flight).
  __device__ __forceinline__ int page(int p) const {
    typedef __attribute__((address_space(4))) const int32_t const_i32;
    return ((const_i32*)table)[p];
  }
  __device__ __forceinline__ size_t at(int page_id, int slot) const {
    return (size_t)page_id * block_stride + (size_t)slot * D;
  }
};

// ---------------------------------------------------------------------------
// LDS layout of one staged K/V tile (64 keys): k_off(mt, ks) is the A-operand
// read of K rows 32*mt + l32 at d = 16*ks + 8*half; v_off(r, dt) the
// transposing read of the V slice starting at row r (r a multiple of 8),
// d tile dt (see pf_pv).
// ---------------------------------------------------------------------------
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

// Q of the items: the rows of waves [4*part, 4*part + 4) of one item fill
// one stage, wave slot w4 (32 rows x D) at w4 * 32 * D, 16-byte chunk c of
// row r at chunk c ^ (r mod D/8) (the B-operand reads of 16 rows then hit
// distinct banks).  Each wave reads its own slot into the Q^T fragments.
// The lane index is made opaque to the compiler in the helpers used at item
// boundaries: their per-lane address arithmetic is then recomputed at each
// use instead of being kept live (or spilled) across the item loop.
__device__ __forceinline__ int opaque_lane() {
  int l = threadIdx.x & 63;
  asm volatile("" : "+v"(l));
  return l;
}

template <int D>
__device__ __forceinline__ void pf_read_q(PfState<D>& st, const bf16_t* __restrict__ slot) {
  constexpr int kSwz = D / 8 - 1;
  const int lane = opaque_lane();
  const int r = lane & 31, half = lane >> 5;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
    st.qf[ks] = *reinterpret_cast<const bf16x8*>(slot + r * D + 8 * ((2 * ks + half) ^ (r & kSwz)));
}

template <int D>
__device__ __forceinline__ void pf_reset(PfState<D>& st) {
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) st.oacc[dt][j] = 0.f;
  st.m_used = -INFINITY;
  st.l = 0.f;
}

// Normalise and store this wave's rows and their log-sum-exp.  The O^T
// accumulators hold, per lane, one row and scattered groups of four d values,
// so the tile goes through this wave's 32 x D/2 slice of LDS, one half of the
// columns at a time (16-byte chunk c of a half row r at chunk c ^ (r mod
// D/16)), and leaves as whole half rows, each D/16-lane group of a store
// instruction writing one contiguous 128-byte (D = 128) piece of a row.
template <int D>
__device__ __forceinline__ void pf_store(const PfState<D>& st, bf16_t* __restrict__ o,
                                         size_t o_stride, float* __restrict__ lse, int r0,
                                         int nq, float scale, bf16_t* __restrict__ slot) {
  constexpr int kHalf = D / 2;                  // columns per pass
  constexpr int kCh = kHalf / 8;                // 16-byte chunks per half row
  constexpr int kRowsPerInstr = 64 / kCh;
  constexpr int kSwz = kCh - 1;
  constexpr int kDtHalf = D / 64;               // 32-column tiles per pass
  const int lane = opaque_lane();
  const int half = lane >> 5, r = lane & 31;
  const float lt = st.l + wave_xor(st.l, 32);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
#pragma unroll
  for (int hf = 0; hf < 2; ++hf) {
#pragma unroll
    for (int dl = 0; dl < kDtHalf; ++dl) {
      const int dt = hf * kDtHalf + dl;
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int c = 4 * dl + g4;              // chunk of d = 32*dt + 8*g4 + 4*half in the pass
        const bf16x4 w = to_bf16x4(st.oacc[dt][4 * g4] * inv, st.oacc[dt][4 * g4 + 1] * inv,
                                   st.oacc[dt][4 * g4 + 2] * inv, st.oacc[dt][4 * g4 + 3] * inv);
        *reinterpret_cast<bf16x4*>(slot + r * kHalf + 8 * (c ^ (r & kSwz)) + 4 * half) = w;
      }
    }
    wave_lds_sync();
    // all reads first (one wait), then the stores of the rows that exist
    constexpr int kN = 32 / kRowsPerInstr;
    u32x4 v[kN];
    const int rl = lane / kCh, c = lane % kCh;
#pragma unroll
    for (int i = 0; i < kN; ++i) {
      const int rr = kRowsPerInstr * i + rl;
      v[i] = *reinterpret_cast<const u32x4*>(slot + rr * kHalf + 8 * (c ^ (rr & kSwz)));
    }
    bf16_t* const ol = o + (size_t)(r0 + rl) * o_stride + hf * kHalf + 8 * c;
#pragma unroll
    for (int i = 0; i < kN; ++i)
      if (r0 + kRowsPerInstr * i + rl < nq)
        *reinterpret_cast<u32x4*>(ol + (size_t)(kRowsPerInstr * i) * o_stride) = v[i];
    wave_lds_sync();
  }
  const int row = r0 + r;
  if (lse != nullptr && half == 0 && row < nq)
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
// Software-pipelined tile loop (K/V DMA-staged into four LDS stages of
// ChunkLayout; KV is DenseKV or PagedDmaKV).
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
// steps -- step i takes the exponentials of step i's scores, forms the
// exponent arguments of step i+1's and packs and sums step i-1's -- so no
// vector instruction waits on the one before it (a wave issues in order, and
// such a wait would hold back its next MFMA too).  (Of the orders measured,
// exponentials first after the QK MFMA was fastest by ~0.5%; raising the
// wave priority around the MFMA cost 4-5%.)  A scheduling barrier after each
// step and empty asm statements on the values each step produces keep the
// compiler from regrouping the work (left alone it clusters the MFMAs, and
// the two units take turns).
// `hook(i)` runs at the start of step i (the steady loop issues the next
// tile's copies through it, one instruction every other step).
struct PfNoHook {
  __device__ __forceinline__ void operator()(int) const {}
};
template <int D, int HK, int HV, class Hook = PfNoHook>
__device__ __forceinline__ float pf_full_slot(PfState<D>& st, const ChunkLayout<D>& lay,
                                              const bf16_t* __restrict__ kst,
                                              const bf16_t* __restrict__ vstage,
                                              const f32x16& s_cur, f32x16& s_next,
                                              bf16x8 (&p_cur)[2], const bf16x8 (&p_prev)[2],
                                              float c, float nm, const Hook& hook = Hook()) {
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
    hook(i);
    __builtin_amdgcn_sched_barrier(0);
    acc = mfma32(ka[i], st.qf[i], acc);
    expo(i);
    if (i + 1 < kSteps) arg(i + 1);
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

// What the items of one workgroup share: the sequence, the GQA head group
// and the output.  Items are query tiles of that sequence (item k starts at
// query row q0_of(k)); wave w owns head h0 + w % hw and the 32 rows starting
// at q0 + 32 * (w / hw) of every item.
struct PfGroup {
  const bf16_t* q;     // row 0 of the sequence, head h0
  bf16_t* o;           // row 0 of the sequence, head h0
  float* lse;          // [head][row] from head h0, row 0 (null: none)
  size_t q_stride;     // elements between rows of q and o
  size_t lse_stride;   // elements between heads of lse
  int hw;              // q heads per workgroup
  int nq, nk;          // query rows and keys of the sequence
  int wg_rows;         // rows of an item (a query tile)
  int causal;
  float scale;
};

// ---------------------------------------------------------------------------
// The items of one workgroup, one after another, each over the pipelined
// tile loop above, with the work at an item boundary overlapped:
//   * the next item's Q (two stages: waves 0-3, waves 4-7) and its first K/V
//     tile are copied into LDS in the last three tiles of the current item,
//     each into the stage the current item has just retired (so the HBM
//     latency of Q is hidden behind the current item's compute);
//   * the current item's output leaves (through LDS) between the requests
//     of the next item's tiles 1 and 2, and is not waited for.
// Rows past the sequence end are read from its last row (finite data; those
// rows are never stored).
// ---------------------------------------------------------------------------
template <int D, int W, class KV, class Q0Of>
__device__ __forceinline__ void prefill_items(const PfGroup& g, const KV& kv, const Q0Of& q0_of,
                                              int n_items, bf16_t* __restrict__ s0,
                                              bf16_t* __restrict__ s1, bf16_t* __restrict__ s2,
                                              bf16_t* __restrict__ s3) {
  using Lay = ChunkLayout<D>;
  constexpr int kCh = D / 8;                     // 16-byte chunks per row
  constexpr int kInstr = kPfBN * kCh / (64 * W);  // K (and V) DMA instructions per wave per tile
  static_assert(kInstr >= 1 && (kPfBN * kCh) % (64 * W) == 0, "tile staging layout");
  constexpr int kLoadsPerTile = 2 * kInstr;      // vmcnt events per wave per tile
  static_assert(2 * kLoadsPerTile < 64, "vmcnt range");
  static_assert(W == 8, "Q staging: two stages of four waves");
  static_assert(4 * 32 * D == Lay::kElemsTile, "a stage holds the Q rows of four waves");
  // a Q stage takes as many DMA instructions per wave as a K/V tile
  static_assert(4 * 32 * kCh == 64 * W * kLoadsPerTile, "Q staging instruction count");
  const int tid = threadIdx.x;
  const int wave = wave_id(), lane = tid & 63;
  const int nq = g.nq, nk = g.nk;
  const int rb = wave / g.hw;                    // this wave's row block
  const int hoff = (wave % g.hw) * D;            // this wave's head

  // ---- DMA helpers ----------------------------------------------------------
  // K/V tile: instruction i of this wave writes staged chunks [64*gi, 64*gi +
  // 64) of the K and of the V region, gi = wave*kInstr + i; lane l fetches the
  // (row, chunk) that staged chunk 64*gi + l holds.  Rows past the sequence
  // end are loaded from its last row (finite data; those keys are masked --
  // the tail slots of a cache page may hold anything).  The 16 rows of one
  // instruction lie in one page: for a paged cache its id is read once for
  // the wave, from ids loaded while the previous tile was issued.
  static_assert(kPfBN == 64, "a tile spans four pages");
  const int last_page = (nk - 1) >> 4;
  int pid0 = 0, pid1 = 0, pid2 = 0, pid3 = 0;   // page ids of the next tile issued
  auto load_ids = [&](int k0) {
    if constexpr (KV::kPaged) {
      const int p0 = k0 >> 4;
      pid0 = kv.page(min(p0, last_page));
      pid1 = kv.page(min(p0 + 1, last_page));
      pid2 = kv.page(min(p0 + 2, last_page));
      pid3 = kv.page(min(p0 + 3, last_page));
    }
  };
  auto pick = [&](int qi) {   // qi wave-uniform, 0..3; selects values, not lvalues
    const int lo = (qi & 1) ? pid1 : pid0;   // (selecting lvalues would put the
    const int hi = (qi & 1) ? pid3 : pid2;   // four ids in private memory)
    return (qi & 2) ? hi : lo;
  };
  // Full tiles of dense K/V: per-lane byte offsets of the first instruction,
  // computed once; instruction i then adds 64*i bytes (K) or 16*i rows (V),
  // folded into the scalar base.  (The pattern holds for D = 64 and
  // 128 with eight waves: the chunks of instruction i are those of
  // instruction 0 moved by four chunks of the same rows (K) or by 16 rows (V).)
  // For a paged cache the rows of one instruction are the 16 slots of one
  // page, so the per-lane offset is within the page (slot r % 16) and the
  // page's base is the scalar part.
  static_assert(kInstr == 1 || kInstr == 2, "full-tile copy");
  uint32_t k_off0 = 0, v_off0 = 0;
  {
    int kr, kc, vr, vc;
    Lay::k_src(64 * wave * kInstr + lane, kr, kc);
    Lay::v_src(64 * wave * kInstr + lane, vr, vc);
    if constexpr (KV::kPaged) {
      k_off0 = (uint32_t)(((kr & 15) * D + kc * 8) * sizeof(bf16_t));
      v_off0 = (uint32_t)(((vr & 15) * D + vc * 8) * sizeof(bf16_t));
    } else {
      k_off0 = (uint32_t)((kr * kv.stride + kc * 8) * sizeof(bf16_t));
      v_off0 = (uint32_t)((vr * kv.stride + vc * 8) * sizeof(bf16_t));
    }
  }
  auto issue_tile = [&](bf16_t* stage, int k0) {
    if (k0 + kPfBN <= nk) {
      const int g0 = wave * kInstr;
      if constexpr (KV::kPaged) {
        // K rows of instruction 1 are those of instruction 0 (64 bytes on);
        // V rows of instruction i are rows 16*i on (the next page).
        int kr0, vr0, unused;
        Lay::k_src(64 * g0, kr0, unused);
        Lay::v_src(64 * g0, vr0, unused);
        const bf16_t* kb = kv.k + kv.at(pick(kr0 >> 4), 0);
        dma16_s(kb, k_off0, stage + 64 * g0 * 8);
        dma16_s(kv.v + kv.at(pick(vr0 >> 4), 0), v_off0, stage + kPfBN * D + 64 * g0 * 8);
        if constexpr (kInstr == 2) {
          dma16_s(kb + 32, k_off0, stage + 64 * (g0 + 1) * 8);
          dma16_s(kv.v + kv.at(pick((vr0 >> 4) + 1), 0), v_off0,
                  stage + kPfBN * D + 64 * (g0 + 1) * 8);
        }
        load_ids(k0 + kPfBN);
      } else {
        const bf16_t* kb = kv.krow(k0);
        const bf16_t* vb = kv.vrow(k0);
        dma16_s(kb, k_off0, stage + 64 * g0 * 8);
        dma16_s(vb, v_off0, stage + kPfBN * D + 64 * g0 * 8);
        if constexpr (kInstr == 2) {
          dma16_s(kb + 32, k_off0, stage + 64 * (g0 + 1) * 8);    // 64 bytes on
          dma16_s(vb + (size_t)16 * kv.stride, v_off0, stage + kPfBN * D + 64 * (g0 + 1) * 8);
        }
      }
      return;
    }
    const int ln = opaque_lane();
#pragma unroll
    for (int i = 0; i < kInstr; ++i) {
      const int gi = wave * kInstr + i;
      const int p = 64 * gi + ln;
      int kr, kc, vr, vc;
      Lay::k_src(p, kr, kc);
      Lay::v_src(p, vr, vc);
      if constexpr (KV::kPaged) {
        int kr0, vr0, unused;
        Lay::k_src(64 * gi, kr0, unused);
        Lay::v_src(64 * gi, vr0, unused);
        dma16(kv.k + kv.at(pick(kr0 >> 4), min(k0 + kr, nk - 1) & 15) + kc * 8,
              stage + 64 * gi * 8);
        dma16(kv.v + kv.at(pick(vr0 >> 4), min(k0 + vr, nk - 1) & 15) + vc * 8,
              stage + kPfBN * D + 64 * gi * 8);
      } else {
        dma16(kv.krow(min(k0 + kr, nk - 1)) + kc * 8, stage + 64 * gi * 8);
        dma16(kv.vrow(min(k0 + vr, nk - 1)) + vc * 8, stage + kPfBN * D + 64 * gi * 8);
      }
    }
    load_ids(k0 + kPfBN);   // the tile issued next is the following one
  };
  // Instruction `part` (0..3: K, V, K, V) of issue_tile for a tile, in the
  // same order (a paged cache's next page ids are read after the last); a
  // partial tile goes out whole at part 0.
  auto issue_tile_part = [&](bf16_t* stage, int k0, int part) {
    if (k0 + kPfBN > nk) {
      if (part == 0) issue_tile(stage, k0);
      return;
    }
    const int g0 = wave * kInstr;
    if (part >= 2 * kInstr) return;
    if constexpr (KV::kPaged) {
      int kr0, vr0, unused;
      Lay::k_src(64 * g0, kr0, unused);
      Lay::v_src(64 * g0, vr0, unused);
      if (part == 0) dma16_s(kv.k + kv.at(pick(kr0 >> 4), 0), k_off0, stage + 64 * g0 * 8);
      if (part == 1)
        dma16_s(kv.v + kv.at(pick(vr0 >> 4), 0), v_off0, stage + kPfBN * D + 64 * g0 * 8);
      if (part == 2)
        dma16_s(kv.k + kv.at(pick(kr0 >> 4), 0) + 32, k_off0, stage + 64 * (g0 + 1) * 8);
      if (part == 3)
        dma16_s(kv.v + kv.at(pick((vr0 >> 4) + 1), 0), v_off0,
                stage + kPfBN * D + 64 * (g0 + 1) * 8);
      if (part == 2 * kInstr - 1) load_ids(k0 + kPfBN);
    } else {
      const bf16_t* kb = kv.krow(k0);
      const bf16_t* vb = kv.vrow(k0);
      if (part == 0) dma16_s(kb, k_off0, stage + 64 * g0 * 8);
      if (part == 1) dma16_s(vb, v_off0, stage + kPfBN * D + 64 * g0 * 8);
      if (part == 2) dma16_s(kb + 32, k_off0, stage + 64 * (g0 + 1) * 8);
      if (part == 3)
        dma16_s(vb + (size_t)16 * kv.stride, v_off0, stage + kPfBN * D + 64 * (g0 + 1) * 8);
    }
  };
  // Q rows of waves [4*part, 4*part + 4) of the item starting at row q0 (the
  // layout pf_read_q expects).
  auto issue_q = [&](bf16_t* stage, int part, int q0) {
    const int ln = opaque_lane();
#pragma unroll
    for (int i = 0; i < kLoadsPerTile; ++i) {
      const int gi = wave * kLoadsPerTile + i;
      const int p = 64 * gi + ln;
      const int w4 = p / (32 * kCh), rem = p % (32 * kCh);
      const int r = rem / kCh, c = (rem % kCh) ^ (r & (kCh - 1));
      const int w = 4 * part + w4;
      const int qrow = min(q0 + 32 * (w / g.hw) + r, nq - 1);
      dma16(g.q + (size_t)qrow * g.q_stride + (w % g.hw) * D + 8 * c, stage + 64 * gi * 8);
    }
  };
  // Wait until at most `tiles` DMA jobs (K/V tiles or Q stages) of this wave
  // are in flight (vmcnt in bits 3:0 and 15:14; expcnt and lgkmcnt at max).
  auto wait_tiles = [](int tiles) {
    constexpr int k1 = kLoadsPerTile, k2 = 2 * kLoadsPerTile;
    if (tiles >= 2)
      __builtin_amdgcn_s_waitcnt(0x0F70 | (k2 & 15) | ((k2 >> 4) << 14));
    else if (tiles == 1)
      __builtin_amdgcn_s_waitcnt(0x0F70 | (k1 & 15) | ((k1 >> 4) << 14));
    else
      __builtin_amdgcn_s_waitcnt(0x0F70);
  };
  // Key tiles of the item starting at q0 (the workgroup's last row bounds it).
  auto item_tiles = [&](int q0) {
    const int wg_last = min(q0 + g.wg_rows, nq) - 1;
    const int kend = g.causal ? min(nk, wg_last + (nk - nq) + 1) : nk;
    return kend > 0 ? (kend + kPfBN - 1) / kPfBN : 0;
  };
  // Index of the first item at or after k that has rows, or n_items.
  auto next_item = [&](int k) {
#pragma clang loop vectorize(disable) unroll(disable)
    while (k < n_items && q0_of(k) >= nq) ++k;
    return k;
  };

  const Lay lay;
  PfState<D> st;
  bf16_t* prev = s3;
  bf16_t* cur = s0;
  bf16_t* next = s1;
  bf16_t* after = s2;

  int k = next_item(0);
  if (k >= n_items) return;
  int q0 = q0_of(k);
  int nt = item_tiles(q0);
  // ---- first item: Q to s0/s1, tile 0 to s2, tile 1 to s3 -----------------
  issue_q(s0, 0, q0);
  issue_q(s1, 1, q0);
  if (nt > 0) {
    load_ids(0);
    issue_tile(s2, 0);
  }
  if (nt > 1) issue_tile(s3, kPfBN);
  wait_tiles(nt > 1 ? 1 : 0);
  pf_barrier();
  pf_read_q(st, (wave < 4 ? s0 : s1) + (wave & 3) * 32 * D);
  pf_barrier();                                  // Q read: s0 free
  if (nt > 2) issue_tile(s0, 2 * kPfBN);
  prev = s1;
  cur = s2;
  next = s3;
  after = s0;

  while (true) {
    // ---- one item -------------------------------------------------------
    const int r0 = q0 + 32 * rb;
    const int row = r0 + (lane & 31);
    const PfRange rg = pf_range(nq, nk, q0, g.wg_rows, r0, g.causal);
    PfPipeCtx cx;
    cx.c = g.scale * kLog2e;
    cx.nbw = (rg.kend_w + 31) >> 5;
    cx.lim = g.causal ? min(nk - 1, row + rg.off) : nk - 1;
    cx.mlim = g.causal ? min(nk - 1, r0 + rg.off) : nk - 1;
    pf_reset(st);
    const int k_next = next_item(k + 1);
    const bool has_next = k_next < n_items;
    const int q0n = has_next ? q0_of(k_next) : 0;
    const int ntn = has_next ? item_tiles(q0n) : 0;
    // DMA jobs for the next item, issued as stages retire: 0 = Q of waves
    // 0-3, 1 = Q of waves 4-7, 2 = its first K/V tile (none if it has no
    // keys).  Job j goes to the stage that is cur, next, after (j = 0, 1, 2)
    // once the loop has ended: the stage of tile nt-4+j, retired at tile
    // nt-3+j, where the loop issues it (jobs whose tile is before 0 are
    // issued after the loop).  `jobs` counts those issued, for the waits.
    int jobs = 0;
    auto issue_job = [&](bf16_t* stage, int j) {
      if (j < 2)
        issue_q(stage, j, q0n);
      else if (ntn > 0) {
        load_ids(0);
        issue_tile(stage, 0);
      } else {
        return;
      }
      ++jobs;
    };

    // An item of one or two key tiles leaves stages unused (after; next too
    // for one tile): the next item's Q goes there now, where the loop end
    // would have put it, instead of after the loop with nothing to hide it.
    bool early0 = false, early1 = false;
    if (has_next && nt == 1) {
      issue_job(next, 0);
      issue_job(after, 1);
      early0 = early1 = true;
    } else if (has_next && nt == 2) {
      issue_job(after, 0);
      early0 = true;
    }

    f32x16 sE = {}, sO = {};
    bf16x8 pE[2] = {}, pO[2] = {};
    if (cx.nbw > 0) {
      // The first block's row maximum is the exponent reference from the
      // start (key 0 is visible to every row): its weights then never need
      // the exact path, which would form them twice.
      sE = pf_qk<D, 0>(st, lay, cur);
      if (31 > cx.mlim) pf_mask(sE, 0, cx.lim);
      float tmax = sE[0];
#pragma unroll
      for (int j = 1; j < 16; ++j) tmax = fmaxf(tmax, sE[j]);
      st.m_used = max_halves(tmax);
    }

    auto rotate = [&]() {
      bf16_t* const retired = prev;
      prev = cur;
      cur = next;
      next = after;
      after = retired;
    };
    // Any tile: slots decide per block what to do (first and last blocks,
    // masks, DMA near the end).  Tile t needs tile t+1 in LDS after the
    // first slot; issued after it are tile t+2 (if any) and the next item's
    // jobs of the tiles before t.
    auto general_step = [&](int t) {
      pf_slot<D, 1, 1>(st, lay, cx, 2 * t, sE, sO, pE, pO, cur, prev);
      wait_tiles((t + 2 < nt ? 1 : 0) + jobs);
      pf_barrier();
      if (t + 3 < nt)
        issue_tile(prev, (t + 3) * kPfBN);
      else if (has_next)
        issue_job(prev, t + 3 - nt);
      pf_slot<D, 0, 0>(st, lay, cx, 2 * t + 1, sO, sE, pO, pE, next, cur);
    };
    // A tile whose two slots are full and unmasked for every wave and whose
    // DMA is due: straight-line code (a separate loop, so that its values
    // never meet the general path's at a join, which would cost register
    // copies).
    auto steady_step = [&](int t) {
      float sum = pf_full_slot<D, 1, 1>(st, lay, cur, prev, sE, sO, pE, pO, cx.c,
                                        -st.m_used * cx.c);
      if (__builtin_expect(wave_any(!(sum <= kPfSumBound)), 0))
        sum = pf_reref(st, sE, cx.c, pE);
      st.l += sum;
      wait_tiles(1);
      pf_barrier();
      // The copies of tile t+3 go out one instruction every other step of
      // the slot rather than all at once: their LDS writes then interleave
      // with the slot's LDS reads instead of arriving as one burst.
      bf16_t* const dst = prev;
      const int k3 = (t + 3) * kPfBN;
      sum = pf_full_slot<D, 0, 0>(st, lay, next, cur, sO, sE, pO, pE, cx.c, -st.m_used * cx.c,
                                  [&](int i) {
                                    if ((i & 1) == 0) issue_tile_part(dst, k3, i >> 1);
                                  });
      if (__builtin_expect(wave_any(!(sum <= kPfSumBound)), 0))
        sum = pf_reref(st, sO, cx.c, pO);
      st.l += sum;
    };
    // Steady tiles are [1, t_end): the item's first row block has the fewest
    // visible keys, so its limits bind every wave.  Tile t needs blocks up to
    // 2t+2 computed (2t+2 < nbw), keys up to 64t+63 unmasked and the DMA of
    // tile t+3 to exist.
    int t_end;
    {
      const int kend0 = g.causal ? min(nk, min(q0 + 32, nq) + rg.off) : nk;
      const int nbw0 = (kend0 + 31) >> 5;
      const int mlim0 = g.causal ? min(nk - 1, q0 + rg.off) : nk - 1;
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

    bf16_t* const o_w = g.o + hoff;
    float* const lse_w = g.lse ? g.lse + (size_t)(wave % g.hw) * g.lse_stride : nullptr;
    if (!has_next) {
      // Every tile before the last has been retired by the last barrier:
      // cur is free for the output.
      pf_store(st, o_w, g.q_stride, lse_w, r0, nq, g.scale, cur + wave * 16 * D);
      return;
    }
    // ---- item boundary ------------------------------------------------------
    // The next item's jobs the loop did not issue (those of tiles before 0)
    // go out now; the stages of tiles before nt-1 were retired by the last
    // barrier.
    if (nt < 3 && !early0) issue_job(cur, 0);
    if (nt < 2 && !early1) issue_job(next, 1);
    if (nt < 1) issue_job(after, 2);
    wait_tiles(0);
    pf_barrier();                                // its Q and first tile are in LDS
    // The Q^T fragments are free (the last product with them is done); the
    // output accumulators are untouched by the read.
    pf_read_q(st, (wave < 4 ? cur : next) + (wave & 3) * 32 * D);
    pf_barrier();                                // Q read, last PV done: cur, next, prev free
    // Tile 1 goes out before the output stores and tile 2 after them.  The
    // next item's first wait leaves one tile's copies in flight, and the
    // vector-memory counter does not tell copies from stores: with the
    // stores issued last, that wait also had to see tile 2 or the stores
    // complete; issued between the tiles, only tile 2 stays in flight.
    if (ntn > 1) issue_tile(prev, kPfBN);
    pf_store(st, o_w, g.q_stride, lse_w, r0, nq, g.scale, cur + wave * 16 * D);
    if (ntn > 2) issue_tile(next, 2 * kPfBN);
    // next item's stages: tile 0 in after, tile 1 in prev, tile 2 in next;
    // cur (the output staging) receives tile 3.
    bf16_t* const st_out = cur;
    cur = after;
    after = next;
    next = prev;
    prev = st_out;
    k = k_next;
    q0 = q0n;
    nt = ntn;
  }
}

// One query tile (a single item), for the chunked-prefill pieces of the mixed
// launch.
template <int D, int W, class KV>
__device__ __forceinline__ void prefill_tile_pipe(const PfGroup& g, const KV& kv, int q0,
                                                  bf16_t* __restrict__ s0, bf16_t* __restrict__ s1,
                                                  bf16_t* __restrict__ s2,
                                                  bf16_t* __restrict__ s3) {
  prefill_items<D, W, KV>(g, kv, [q0](int) { return q0; }, 1, s0, s1, s2, s3);
}

}  // namespace rag
