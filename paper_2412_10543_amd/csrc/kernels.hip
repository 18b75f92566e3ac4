// gfx950 kernels of the RAG-synthesis attention path and their launchers:
//   prefill_varlen_kernel  packed variable-length prefill (dense K/V)
//   paged_decode_kernel    decode rows against a paged KV cache (split-KV
//                          partials are merged inside it by the last split
//                          of each sequence to finish)
//   mixed_kernel           decode rows and chunked-prefill pieces of a
//                          paged cache in one launch
#include <algorithm>
#include <climits>
#include <cstdlib>

#include "common.h"
#include "decode_unit.h"
#include "launch.h"
#include "prefill_tile.h"

namespace rag {

// ---------------------------------------------------------------------------
// Work order of prefill tiles.  A "stream" is one (sequence, kv head) pair;
// all q heads of its GQA group and all its query tiles read the same K/V.  A
// workgroup takes up to four of the group's q heads (a head group) and a set
// of `items` query tiles of one stream, which it runs one after another
// (prefill_items overlaps each tile's start with the end of the one before).
// The tiles of a stream are dealt to its `per` workgroups in a snake order --
// workgroup j takes tiles j, 2*per-1-j, 2*per+j, ... -- so that under the
// causal mask, where tile t costs t+1 key tiles, every workgroup of a stream
// gets nearly the same work.  Stream sigma runs on XCD sigma % 8, so every XCD
// gets the same mix of sequences (and, with 8 kv heads, exactly one kv head
// of each); on an XCD the workgroups of a stream are consecutive, so those
// resident at one time share K/V tiles through its L2.
// ---------------------------------------------------------------------------
#ifndef RAG_PF_WG_PER_CU
#define RAG_PF_WG_PER_CU 32
#endif
constexpr int kPfWgPerCu = RAG_PF_WG_PER_CU;  // workgroups per CU aimed at (load balance)
constexpr int kPfCus = 256;
constexpr int kPfMaxItems = 32;

struct TileCoord {
  int seq, kvh, h0, j;
  bool valid;
};

// Workgroup -> (stream, head group, workgroup j of the stream).
__device__ __forceinline__ TileCoord prefill_coord(int block, int num_streams, int hkv,
                                                   int group, int per) {
  const int hw = pf_heads_per_wg(group);
  const int ng = group / hw;
  int xcd, local;
  xcd_slot(block, xcd, local);
  const int hg = local % ng;
  const int rest = local / ng;
  TileCoord t;
  t.j = rest % per;
  const int stream = xcd + kNumXcd * (rest / per);
  t.valid = stream < num_streams;
  t.seq = stream / hkv;
  t.kvh = stream % hkv;
  t.h0 = t.kvh * group + hg * hw;
  return t;
}

// Query tile of item k of workgroup j (snake order over the per workgroups).
__device__ __forceinline__ int snake_tile(int j, int k, int per) {
  return (k & 1) ? (k + 1) * per - 1 - j : k * per + j;
}

// Items per workgroup and workgroups per (stream, head group) for a launch.
struct PfSplit {
  int items, per, n_qt;
};
// RAG_ATTN_PF_ITEMS=n (read at each launch) fixes the query tiles per
// workgroup at n instead of the load-balancing choice below: a testing and
// tuning knob (every tile is computed the same way whichever workgroup runs
// it, so outputs are bit-identical for any n).
static int pf_items_override() {
  const char* e = std::getenv("RAG_ATTN_PF_ITEMS");
  if (e == nullptr || e[0] == 0) return 0;
  const int n = std::atoi(e);
  return n >= 1 ? std::min(n, kPfMaxItems) : 0;
}

static PfSplit pf_split(int num_seqs, int hkv, int group, int max_seqlen_q, bool multi) {
  const int rows = pf_rows_per_tile(group, kPfWavesDense);
  PfSplit p;
  p.n_qt = (max_seqlen_q + rows - 1) / rows;
  const int64_t streams = (int64_t)num_seqs * hkv * (group / pf_heads_per_wg(group));
  if (!multi || p.n_qt <= 1) {
    p.items = 1;
    p.per = p.n_qt;
    return p;
  }
  if (const int forced = pf_items_override()) {
    p.items = std::min(forced, p.n_qt);
    p.per = (p.n_qt + p.items - 1) / p.items;
    return p;
  }
  const int64_t want = (int64_t)kPfWgPerCu * kPfCus;
  const int64_t per = std::max<int64_t>(1, (want + streams - 1) / std::max<int64_t>(streams, 1));
  int items = (int)std::min<int64_t>(kPfMaxItems, (p.n_qt + per - 1) / per);
  items = std::max(1, items);
  p.items = items;
  p.per = (p.n_qt + items - 1) / items;
  return p;
}

static int64_t tile_grid(int num_seqs, int hkv, int group, const PfSplit& sp) {
  const int64_t streams = (int64_t)num_seqs * hkv;
  const int64_t per_xcd = (streams + kNumXcd - 1) / kNumXcd;
  return (int64_t)kNumXcd * per_xcd * sp.per * (group / pf_heads_per_wg(group));
}

int64_t prefill_grid(int num_seqs, int hkv, int group, int max_seqlen_q) {
  return tile_grid(num_seqs, hkv, group, pf_split(num_seqs, hkv, group, max_seqlen_q, true));
}

int64_t paged_prefill_grid(int num_pieces, int hkv, int group, int max_seqlen_q) {
  return tile_grid(num_pieces, hkv, group, pf_split(num_pieces, hkv, group, max_seqlen_q, false));
}

int64_t paged_decode_grid(int num_decode, int hkv, int num_splits) {
  return (int64_t)num_decode * hkv * num_splits;
}

// Paged KV-cache write fused into the prompt prefill: the K and V rows
// [r0, r1) of one (sequence, kv head) stream go to their slots in the paged
// cache (slot = page * 16 + offset; a negative slot skips the row).  Run by
// each workgroup after its last item, for the key rows of its own query
// tiles, so every row of a sequence is written once; the rows were streamed
// through this XCD's L2 by the prefill itself.
template <int D>
__device__ __forceinline__ void prefill_rows_to_cache(const bf16_t* __restrict__ k,
                                                      const bf16_t* __restrict__ v,
                                                      size_t stride, bf16_t* __restrict__ kc,
                                                      bf16_t* __restrict__ vc,
                                                      size_t block_stride,
                                                      const int32_t* __restrict__ slots,
                                                      int r0, int r1) {
  constexpr int kCh = D / 8;
  const int n = (r1 - r0) * kCh;
  for (int p = threadIdx.x; p < n; p += 64 * kPfWavesDense) {
    const int r = r0 + p / kCh, c = p % kCh;
    const int slot = slots[r];
    if (slot < 0) continue;
    const size_t src = (size_t)r * stride + c * 8;
    const size_t dst = (size_t)(slot >> 4) * block_stride + (size_t)(slot & 15) * D + c * 8;
    const u32x4 kx = load16(k + src);
    const u32x4 vx = load16(v + src);
    *reinterpret_cast<u32x4*>(kc + dst) = kx;
    *reinterpret_cast<u32x4*>(vc + dst) = vx;
  }
}

template <int D>
__global__ __launch_bounds__(64 * kPfWavesDense, 2) void prefill_varlen_kernel(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k,
    const bf16_t* __restrict__ v, bf16_t* __restrict__ o, float* __restrict__ lse,
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_k, int num_seqs,
    int hq, int hkv, int items, int per, float scale, int causal,
    bf16_t* __restrict__ k_cache, bf16_t* __restrict__ v_cache,
    const int32_t* __restrict__ slots) {
  // four K/V stages (separate arrays: the compiler then knows a DMA write to
  // one stage never aliases an LDS read of another)
  __shared__ __attribute__((aligned(16))) bf16_t st0[ChunkLayout<D>::kElemsTile];
  __shared__ __attribute__((aligned(16))) bf16_t st1[ChunkLayout<D>::kElemsTile];
  __shared__ __attribute__((aligned(16))) bf16_t st2[ChunkLayout<D>::kElemsTile];
  __shared__ __attribute__((aligned(16))) bf16_t st3[ChunkLayout<D>::kElemsTile];
  const int group = hq / hkv;
  const TileCoord tc = prefill_coord(blockIdx.x, num_seqs * hkv, hkv, group, per);
  if (!tc.valid) return;
  const int qb = cu_q[tc.seq], nq = cu_q[tc.seq + 1] - qb;
  const int kb = cu_k[tc.seq], nk = cu_k[tc.seq + 1] - kb;
  const int rows = pf_rows_per_tile(group, kPfWavesDense);
  if (tc.j * rows >= nq) return;
  const int tq = cu_q[num_seqs];
  PfGroup g;
  g.q = q + ((size_t)qb * hq + tc.h0) * D;
  g.o = o + ((size_t)qb * hq + tc.h0) * D;
  g.lse = lse ? lse + (size_t)tc.h0 * tq + qb : nullptr;
  g.q_stride = (size_t)hq * D;
  g.lse_stride = (size_t)tq;
  g.hw = pf_heads_per_wg(group);
  g.nq = nq;
  g.nk = nk;
  g.wg_rows = rows;
  g.causal = causal;
  g.scale = scale;
  DenseKV kv{k + ((size_t)kb * hkv + tc.kvh) * D, v + ((size_t)kb * hkv + tc.kvh) * D,
             (size_t)hkv * D};
  const int j = tc.j;
  prefill_items<D, kPfWavesDense, DenseKV>(
      g, kv, [j, per, rows](int it) { return snake_tile(j, it, per) * rows; }, items, st0, st1,
      st2, st3);
  // Fused cache write (prompt prefill: query rows are the key rows): the
  // first head group of the kv head writes the key rows of its query tiles.
  if (slots != nullptr && tc.h0 == tc.kvh * group) {
    const size_t block_stride = (size_t)hkv * 16 * D;
    for (int it = 0; it < items; ++it) {
      const int q0 = snake_tile(j, it, per) * rows;
      if (q0 >= nq) continue;
      prefill_rows_to_cache<D>(kv.k, kv.v, kv.stride, k_cache + (size_t)tc.kvh * 16 * D,
                               v_cache + (size_t)tc.kvh * 16 * D, block_stride, slots + kb, q0,
                               min(q0 + rows, nk));
    }
  }
}

// ---------------------------------------------------------------------------
// Paged kernel.  In a mixed batch the grid holds n_pf_blocks chunked-prefill
// tiles and the decode units, interleaved in groups of eight consecutive
// blocks (all tiles or all units; tile groups spread evenly through the grid)
// so that MFMA-bound tiles and HBM-bound units share the CUs instead of
// running one after the other; a tile keeps its XCD (block % 8).  Decode
// unit u is split sp = u / (num_decode * hkv) of (sequence, kv head)
// u % (num_decode * hkv), where split sp of a sequence with P pages is the
// page range [sp * pps, min((sp + 1) * pps, P)).
// ---------------------------------------------------------------------------
struct PagedKernelArgs {
  const bf16_t* q;
  const bf16_t* kc;
  const bf16_t* vc;
  bf16_t* o;
  const int32_t* tables;
  const int32_t* kv_lens;
  const int32_t* cu_q;
  float* part_o;
  float* part_lse;
  int* arrivals;              // one counter per (decode sequence, kv head)
  const bf16_t* k_new;        // appended tokens [num_decode, hkv, D] (append launch only)
  const bf16_t* v_new;
  int num_seqs, num_decode, max_blocks, hq, hkv, num_splits, pps;
  int slots;                  // partial-result slots per (row, head): workspace stride
  int bal_units;              // balanced decode: units per kv head (0: uniform splits)
  int n_pf_blocks, n_qt;
  int n_dec_groups;           // mixed batches: groups of eight decode units
  float scale;
};

// One piece of a decode row: pages [p_begin, p_end) of (row s, kv head kvh),
// split sp of n_sp, on W waves taking NP pages a step.
template <int D, int NP, int W, bool kAppend = false>
__device__ __forceinline__ void decode_piece(const PagedKernelArgs& a, int group,
                                             size_t block_stride, int s, int kvh, int kv_len,
                                             int p_begin, int p_end, int sp, int n_sp,
                                             bf16_t* lds) {
  const int row = a.cu_q ? a.cu_q[s] : s;
  const int h0 = kvh * group;
  DecodeOut out;
  out.o = a.o + ((size_t)row * a.hq + h0) * D;
  out.part_o = a.part_o ? a.part_o + (size_t)s * a.hq * a.slots * D + (size_t)h0 * a.slots * D
                        : nullptr;
  out.part_lse = a.part_lse ? a.part_lse + ((size_t)s * a.hq + h0) * a.slots : nullptr;
  out.arrival = a.arrivals ? a.arrivals + (size_t)s * a.hkv + kvh : nullptr;
  out.sp = sp;
  out.n_sp = n_sp;
  out.num_splits = a.slots;
  const size_t nrow = ((size_t)s * a.hkv + kvh) * D;
  decode_unit<D, NP, W, kAppend>(a.q + ((size_t)row * a.hq + h0) * D,
                                 a.kc + (size_t)kvh * 16 * D, a.vc + (size_t)kvh * 16 * D,
                                 block_stride, a.tables + (size_t)s * a.max_blocks, kv_len, group,
                                 p_begin, p_end, a.scale, out, lds,
                                 kAppend ? a.k_new + nrow : nullptr,
                                 kAppend ? a.v_new + nrow : nullptr);
}

// Decode unit u with fixed page ranges (see above), on W waves.
template <int D, int NP, int W, bool kAppend = false>
__device__ __forceinline__ void decode_block(const PagedKernelArgs& a, int u, int group,
                                             size_t block_stride, bf16_t* lds) {
  const int64_t pairs = (int64_t)a.num_decode * a.hkv;
  if ((int64_t)u >= pairs * a.num_splits) return;
  const int sp = (int)(u / pairs);
  const int pr = (int)(u % pairs);
  const int s = pr / a.hkv, kvh = pr % a.hkv;
  const int kv_len = min(a.kv_lens[s], a.max_blocks * 16);
  const int n_pages = (kv_len + 15) >> 4;
  const int n_sp = (n_pages + a.pps - 1) / a.pps;
  if (sp >= n_sp && sp > 0) return;
  const int p_begin = sp * a.pps;
  const int p_end = min(n_pages, p_begin + a.pps);
  decode_piece<D, NP, W, kAppend>(a, group, block_stride, s, kvh, kv_len, p_begin, p_end, sp,
                                  n_sp, lds);
}

// Balanced decode units: the pages of all rows of one kv head, laid end to
// end (row by row), are cut into equal ranges of at least kDecMinPages pages
// (at most bal_units of them); unit k of kv head kvh attends the pieces of the
// rows its range covers (usually one or two), each piece split sp of the n_sp
// units that cover its row.  Unit sizes no longer follow the rows' lengths,
// so every CU streams the same number of pages and none is left with a long
// tail.  The plan comes from kv_lens, loaded once (one lane per row, rows in
// chunks of 64; fewer than 256 rows take this path) and walked with
// wave-uniform reads.
constexpr int kBalMaxChunks = 4;

template <int D, int NP, int W, bool kAppend>
__device__ __forceinline__ void decode_block_balanced(const PagedKernelArgs& a, int u, int group,
                                                      size_t block_stride, bf16_t* lds) {
  const int kvh = u % a.hkv, k = u / a.hkv;
  if (k >= a.bal_units) return;
  const int S = a.num_decode, lane = threadIdx.x & 63, cap = a.max_blocks * 16;
  int kl[kBalMaxChunks];
#pragma unroll
  for (int c = 0; c < kBalMaxChunks; ++c) {
    const int s = c * kWave + lane;
    kl[c] = s < S ? min(a.kv_lens[s], cap) : 0;
  }
  int total = 0;
#pragma unroll
  for (int c = 0; c < kBalMaxChunks; ++c)
    for (int i = 0; i < min(kWave, S - c * kWave); ++i)
      total += (__builtin_amdgcn_readlane(kl[c], i) + 15) >> 4;
  // at least kDecMinPages pages per unit (short batches use fewer units)
  const int K = max(1, min(a.bal_units, total / kDecMinPages));
  if (k >= K) return;
  // 32-bit arithmetic: the host takes this path only when rows x table
  // width x units stays below 2^31
  const uint32_t ut = (uint32_t)total, uk = (uint32_t)K;
  const int lo = (int)((uint32_t)k * ut / uk), hi = (int)((uint32_t)(k + 1) * ut / uk);
  // unit holding global page g: ceil((g + 1) K / total) - 1
  auto unit_of = [&](int g) { return (int)(((uint32_t)(g + 1) * uk + ut - 1) / ut) - 1; };
  int gs = 0;                 // first global page of the row
  bool first_piece = true;
  // one call site of decode_piece (rows walked in one loop, the chunk of a
  // row picked by value): the kernel's code stays one copy of the unit
  for (int s = 0; s < S && gs < hi; ++s) {
    static_assert(kBalMaxChunks == 4, "row chunk select");
    const int c = s >> 6;
    const int klc = c == 0 ? kl[0] : c == 1 ? kl[1] : c == 2 ? kl[2] : kl[3];
    const int kls = __builtin_amdgcn_readlane(klc, s & 63);
    const int ps = (kls + 15) >> 4;
    if (ps > 0 && gs + ps > lo) {
      const int first = unit_of(gs), last = unit_of(gs + ps - 1);
      if (!first_piece) __syncthreads();   // LDS of the previous piece fully read
      first_piece = false;
      decode_piece<D, NP, W, kAppend>(a, group, block_stride, s, kvh, kls,
                                      max(lo, gs) - gs, min(hi, gs + ps) - gs, k - first,
                                      last - first + 1, lds);
    }
    gs += ps;
  }
}

template <int D, bool kAppend>
__global__ __launch_bounds__(kDecThreads, 2) void paged_decode_balanced_kernel(
    PagedKernelArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t lds[DecLds<D>::kBytes / 2];
  decode_block_balanced<D, kDecPages, kDecWaves, kAppend>(a, blockIdx.x, a.hq / a.hkv,
                                                          (size_t)a.hkv * 16 * D, lds);
}

// Decode rows only: one four-wave workgroup per decode unit.  kAppend: each
// row's last key is the step's new token, taken from k_new / v_new and
// stored into its cache slot by the same launch.
template <int D, bool kAppend>
__global__ __launch_bounds__(kDecThreads, 2) void paged_decode_kernel(PagedKernelArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t lds[DecLds<D>::kBytes / 2];
  decode_block<D, kDecPages, kDecWaves, kAppend>(a, blockIdx.x, a.hq / a.hkv,
                                                 (size_t)a.hkv * 16 * D, lds);
}

// Mixed batch: eight-wave workgroups.  A chunked-prefill tile runs the dense
// prefill's pipelined tile loop with K/V gathered from the paged cache; a
// decode unit runs on all eight waves (a tile workgroup fills the CU's
// registers, so a decode unit has the CU to itself and needs twice the pages
// in flight of a four-wave unit to keep its share of HBM bandwidth).
template <int D>
__global__ __launch_bounds__(64 * kPfWavesDense, 2) void mixed_kernel(PagedKernelArgs a) {
  constexpr int kE = ChunkLayout<D>::kElemsTile;
  using DL = DecLds<D, kMixedDecPages, kPfWavesDense>;
  __shared__ __attribute__((aligned(16))) bf16_t lds[4 * kE > DL::kBytes / 2 ? 4 * kE
                                                                           : DL::kBytes / 2];
  const int group = a.hq / a.hkv;
  const size_t block_stride = (size_t)a.hkv * 16 * D;
  const int64_t tile_groups = a.n_pf_blocks / kNumXcd;
  const int64_t groups = tile_groups + a.n_dec_groups;
  const int gi = blockIdx.x / kNumXcd, x = blockIdx.x % kNumXcd;
  const int tiles_before = (int)((int64_t)gi * tile_groups / groups);
  const bool is_tile = (int64_t)(gi + 1) * tile_groups / groups > tiles_before;
  if (is_tile) {
    const int num_pieces = a.num_seqs - a.num_decode;
    const TileCoord tc = prefill_coord(kNumXcd * tiles_before + x, num_pieces * a.hkv, a.hkv,
                                       group, a.n_qt);
    if (!tc.valid) return;
    const int s = a.num_decode + tc.seq;
    const int qb = a.cu_q[s], nq = a.cu_q[s + 1] - qb;
    const int rows = pf_rows_per_tile(group, kPfWavesDense);
    const int q0 = (a.n_qt - 1 - tc.j) * rows;   // tiles with the most keys first
    if (q0 >= nq) return;
    PfGroup g;
    g.q = a.q + ((size_t)qb * a.hq + tc.h0) * D;
    g.o = a.o + ((size_t)qb * a.hq + tc.h0) * D;
    g.lse = nullptr;
    g.q_stride = (size_t)a.hq * D;
    g.lse_stride = 0;
    g.hw = pf_heads_per_wg(group);
    g.nq = nq;
    g.nk = min(a.kv_lens[s], a.max_blocks * 16);
    g.wg_rows = rows;
    g.causal = 1;
    g.scale = a.scale;
    const PagedDmaKV<D> kv{a.kc + (size_t)tc.kvh * 16 * D, a.vc + (size_t)tc.kvh * 16 * D,
                           a.tables + (size_t)s * a.max_blocks, block_stride};
    prefill_tile_pipe<D, kPfWavesDense, PagedDmaKV<D>>(g, kv, q0, lds, lds + kE, lds + 2 * kE,
                                                       lds + 3 * kE);
    return;
  }
  decode_block<D, kMixedDecPages, kPfWavesDense>(a, kNumXcd * (gi - tiles_before) + x, group,
                                                 block_stride, lds);
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <int D>
static hipError_t launch_prefill_d(const PrefillArgs& a, hipStream_t stream) {
  const int group = a.hq / a.hkv;
  const PfSplit sp = pf_split(a.num_seqs, a.hkv, group, a.max_seqlen_q, true);
  const int64_t grid = tile_grid(a.num_seqs, a.hkv, group, sp);
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(prefill_varlen_kernel<D>, dim3((unsigned)grid), dim3(64 * kPfWavesDense), 0,
                     stream,
                     (const bf16_t*)a.q, (const bf16_t*)a.k, (const bf16_t*)a.v, (bf16_t*)a.o,
                     a.lse, a.cu_q, a.cu_k, a.num_seqs, a.hq, a.hkv, sp.items, sp.per, a.scale,
                     a.causal, (bf16_t*)a.k_cache, (bf16_t*)a.v_cache, a.slots);
  return hipGetLastError();
}

hipError_t launch_prefill_varlen(const PrefillArgs& a, hipStream_t stream) {
  return a.d == 64 ? launch_prefill_d<64>(a, stream) : launch_prefill_d<128>(a, stream);
}

template <int D>
static hipError_t launch_paged_d(const PagedArgs& a, hipStream_t stream) {
  const int group = a.hq / a.hkv;
  PagedKernelArgs k;
  k.q = (const bf16_t*)a.q;
  k.kc = (const bf16_t*)a.k_cache;
  k.vc = (const bf16_t*)a.v_cache;
  k.o = (bf16_t*)a.o;
  k.tables = a.block_tables;
  k.kv_lens = a.kv_lens;
  k.cu_q = a.cu_q;
  k.part_o = a.part_o;
  k.part_lse = a.part_lse;
  k.arrivals = a.arrivals;
  k.k_new = (const bf16_t*)a.k_new;
  k.v_new = (const bf16_t*)a.v_new;
  k.num_seqs = a.num_seqs;
  k.num_decode = a.num_decode;
  k.max_blocks = a.max_blocks;
  k.hq = a.hq;
  k.hkv = a.hkv;
  k.num_splits = a.num_splits;
  k.pps = std::max(1, (a.max_blocks + a.num_splits - 1) / a.num_splits);
  k.slots = std::max(a.slots, a.num_splits);
  k.bal_units = a.cu_q == nullptr ? a.bal_units : 0;
  k.scale = a.scale;
  const bool mixed = a.cu_q != nullptr && a.num_seqs > a.num_decode;
  const int pf_rows = pf_rows_per_tile(group, kPfWavesDense);
  k.n_qt = mixed ? (a.max_seqlen_q + pf_rows - 1) / pf_rows : 0;
  const int64_t pf = mixed ? paged_prefill_grid(a.num_seqs - a.num_decode, a.hkv, group,
                                                a.max_seqlen_q)
                           : 0;
  k.n_pf_blocks = (int)pf;
  int64_t dec = k.bal_units > 0 ? (int64_t)k.bal_units * a.hkv
                                : paged_decode_grid(a.num_decode, a.hkv, a.num_splits);
  if (pf > 0) dec = (dec + kNumXcd - 1) / kNumXcd * kNumXcd;   // whole groups of eight
  k.n_dec_groups = (int)(dec / kNumXcd);
  const int64_t grid = pf + dec;
  if (grid > 0) {
    if (pf > 0)
      hipLaunchKernelGGL(mixed_kernel<D>, dim3((unsigned)grid), dim3(64 * kPfWavesDense), 0,
                         stream, k);
    else if (k.bal_units > 0 && a.k_new != nullptr)
      hipLaunchKernelGGL((paged_decode_balanced_kernel<D, true>), dim3((unsigned)grid),
                         dim3(kDecThreads), 0, stream, k);
    else if (k.bal_units > 0)
      hipLaunchKernelGGL((paged_decode_balanced_kernel<D, false>), dim3((unsigned)grid),
                         dim3(kDecThreads), 0, stream, k);
    else if (a.k_new != nullptr)
      hipLaunchKernelGGL((paged_decode_kernel<D, true>), dim3((unsigned)grid), dim3(kDecThreads),
                         0, stream, k);
    else
      hipLaunchKernelGGL((paged_decode_kernel<D, false>), dim3((unsigned)grid), dim3(kDecThreads),
                         0, stream, k);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_paged(const PagedArgs& a, hipStream_t stream) {
  return a.d == 64 ? launch_paged_d<64>(a, stream) : launch_paged_d<128>(a, stream);
}

}  // namespace rag
