// Ceiling probes for the MI355X (gfx950): what the memory system and the
// matrix cores deliver to kernels shaped like this library's, measured the
// same way (one launch, HIP events around it, by bench.py --ceilings).  They
// compute nothing of the attention method; they bound it:
//   * page reads: 4 KB pages at random places of a multi-GB pool, read with
//     16-byte loads, default or non-temporal policy;
//   * K/V page reads: a K page and a V page per random id, loaded as the
//     paged decode loads them (or both as whole rows, either policy) -- the
//     ceiling of the decode's own access pattern;
//   * stream read: one large contiguous buffer, 16-byte loads, either policy;
//   * MFMA loop: v_mfma_f32_32x32x16_bf16 with independent accumulators, no
//     memory traffic -- the practical bf16 matrix rate;
//   * attention slot: the prefill kernel's own steady 32-key slot (pf_full_slot:
//     QK^T and PV MFMAs, the exp2/FMA/pack/sum vector work of the online
//     softmax, the LDS operand reads) run over and over on two LDS-resident
//     K/V tiles with the per-tile barrier, no copies -- the rate of the inner
//     loop itself;
//   * softmax-MFMA mix: the same MFMA and vector instructions in the same
//     order with the K/V operands in registers (no LDS) -- the rate the
//     instruction mix allows on the matrix core and vector ALU alone;
//   * specialised pairs: the same work split between the two waves of a SIMD
//     (one computes scores and weights for 64 rows, the other PV), the
//     weights passed through LDS -- an alternative layout, for comparison.
// Each workgroup writes one value derived from what it read or computed, so
// nothing is optimised away.  Declared in include/ceiling_probes.h.
#include <hip/hip_runtime.h>

#include "ceiling_probes.h"
#include "common.h"
#include "prefill_tile.h"

namespace rag {
namespace {

// Wave w of workgroup b reads the pages of list entries (b*4 + w)*4 .. +4,
// then the same again one grid further on; a page is 4096 bytes = 4 loads of
// 16 bytes per lane, so every wave has 16 loads (16 KB) in flight per step.
// The load policy is a template parameter: chosen at run time, the compiler
// merges the two loads of the same address and drops the hint.
template <bool kNT>
__device__ __forceinline__ u32x4 probe_load(const u32x4* p) {
  if constexpr (kNT)
    return __builtin_nontemporal_load(p);
  else
    return *p;
}

template <bool kNT>
__global__ __launch_bounds__(256) void probe_pages_kernel(const u32x4* __restrict__ pool,
                                                          const int32_t* __restrict__ ids,
                                                          int64_t n_pages, uint32_t* __restrict__ out) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t stride = (int64_t)gridDim.x * 16;
  uint32_t acc = 0;
  for (int64_t p0 = ((int64_t)blockIdx.x * 4 + w) * 4; p0 < n_pages; p0 += stride) {
    u32x4 v[4][4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t p = min(p0 + j, n_pages - 1);
      const u32x4* base = pool + (size_t)ids[p] * 256;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[j][i] = probe_load<kNT>(base + i * 64 + lane);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc ^= v[j][i][0] ^ v[j][i][1] ^ v[j][i][2] ^ v[j][i][3];
  }
  if (acc == 0x9E3779B9u) out[blockIdx.x] = acc;   // practically never: keeps the loads
}

// The paged decode's own access pattern: per page id, a 4 KB K page and a
// 4 KB V page (two pools), two pages of each per wave and step.  kDecode:
// K loaded as the decode's MFMA operand layout (an instruction takes 64 bytes
// of each of the 16 rows, default policy) and V as four whole 256-byte rows
// per instruction with the non-temporal hint -- the decode kernel's loads;
// otherwise both as whole rows, with the policy kNT.
template <bool kDecode, bool kNT>
__global__ __launch_bounds__(256) void probe_kv_pages_kernel(const u32x4* __restrict__ kpool,
                                                             const u32x4* __restrict__ vpool,
                                                             const int32_t* __restrict__ ids,
                                                             int64_t n_pages,
                                                             uint32_t* __restrict__ out) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int l16 = lane & 15, gq = lane >> 4;
  const int64_t stride = (int64_t)gridDim.x * 8;
  uint32_t acc = 0;
  for (int64_t p0 = ((int64_t)blockIdx.x * 4 + w) * 2; p0 < n_pages; p0 += stride) {
    u32x4 k[2][4], v[2][4];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const size_t id = (size_t)ids[min(p0 + j, n_pages - 1)];
      const u32x4* kb = kpool + id * 256;
      const u32x4* vb = vpool + id * 256;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (kDecode) {
          k[j][i] = probe_load<false>(kb + l16 * 16 + 4 * i + gq);
          v[j][i] = probe_load<true>(vb + i * 64 + lane);
        } else {
          k[j][i] = probe_load<kNT>(kb + i * 64 + lane);
          v[j][i] = probe_load<kNT>(vb + i * 64 + lane);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc ^= k[j][i][0] ^ k[j][i][3] ^ v[j][i][1] ^ v[j][i][2];
  }
  if (acc == 0x9E3779B9u) out[blockIdx.x] = acc;
}

template <bool kNT>
__global__ __launch_bounds__(256) void probe_stream_kernel(const u32x4* __restrict__ buf,
                                                           int64_t n16, uint32_t* __restrict__ out) {
  uint32_t acc = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x * 4;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x * 4 + threadIdx.x; i < n16; i += stride) {
    u32x4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      v[j] = i + j * blockDim.x < n16 ? probe_load<kNT>(buf + i + j * blockDim.x)
                                      : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 4; ++j) acc ^= v[j][0] ^ v[j][1] ^ v[j][2] ^ v[j][3];
  }
  if (acc == 0x9E3779B9u) out[blockIdx.x] = acc;
}

// Four independent 32x32 accumulators per wave, iters k-steps of 4 MFMAs.
__global__ __launch_bounds__(512, 2) void probe_mfma_kernel(int iters, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (lane + i));
    b[i] = (__bf16)(0.002f * (lane - i));
  }
  f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int it = 0; it < iters; ++it) {
    c0 = mfma32(a, b, c0);
    c1 = mfma32(b, a, c1);
    c2 = mfma32(a, a, c2);
    c3 = mfma32(b, b, c3);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 16; ++j) s += c0[j] + c1[j] + c2[j] + c3[j];
  if (s == 1.2345e-30f) out[blockIdx.x] = s;
}

// Per-wave Q fragments and K/V values of the slot probes: small, so every
// block's weights stay near 1 and the exact path runs only at the first block.
__device__ __forceinline__ bf16x8 probe_frag(int lane, int salt) {
  bf16x8 f;
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = (__bf16)(0.01f * (float)(((lane + 3 * i + salt) % 17) - 8));
  return f;
}

// Eight waves (two per SIMD), two 64-key K/V stages filled once; each
// iteration is one tile: slot 2t (K of stage 0, keys 32-63; V of stage 1,
// keys 32-63), the workgroup barrier, slot 2t+1 (K of stage 1, keys 0-31; V
// of stage 0, keys 0-31) -- the steady step of prefill_varlen_kernel without
// its copies.  32 rows x 32 keys x 4 x 128 FLOP per slot and wave.
__global__ __launch_bounds__(512, 2) void probe_attn_slot_kernel(int iters,
                                                                 float* __restrict__ out) {
  constexpr int D = 128;
  using Lay = ChunkLayout<D>;
  __shared__ __attribute__((aligned(16))) bf16_t s0[Lay::kElemsTile];
  __shared__ __attribute__((aligned(16))) bf16_t s1[Lay::kElemsTile];
  for (int i = threadIdx.x; i < Lay::kElemsTile; i += blockDim.x) {
    s0[i] = __builtin_bit_cast(bf16_t, (__bf16)(0.01f * (float)((i % 23) - 11)));
    s1[i] = __builtin_bit_cast(bf16_t, (__bf16)(0.01f * (float)((i % 19) - 9)));
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const Lay lay;
  PfState<D> st;
  pf_reset(st);
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) st.qf[ks] = probe_frag(lane, ks);
  const float c = 0.08838834764831845f * kLog2e;
  f32x16 sE = pf_qk<D, 0>(st, lay, s0), sO = {};
  bf16x8 pE[2] = {}, pO[2] = {};
  float sum = pf_reref(st, sE, c, pE);
  st.l += sum;
  for (int it = 0; it < iters; ++it) {
    sum = pf_full_slot<D, 1, 1>(st, lay, s0, s1, sE, sO, pE, pO, c, -st.m_used * c);
    if (__builtin_expect(wave_any(!(sum <= kPfSumBound)), 0)) sum = pf_reref(st, sE, c, pE);
    st.l += sum;
    pf_barrier();
    sum = pf_full_slot<D, 0, 0>(st, lay, s1, s0, sO, sE, pO, pE, c, -st.m_used * c);
    if (__builtin_expect(wave_any(!(sum <= kPfSumBound)), 0)) sum = pf_reref(st, sO, c, pO);
    st.l += sum;
  }
  float r = st.l;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) r += st.oacc[dt][j];
  if (r == 1.2345e-30f) out[blockIdx.x] = r;
}

// A different split of the same slot work (the layout the prefill does not
// use, measured for comparison): the two waves of a SIMD specialise.  Wave w
// < 4 (the producer of pair w) computes QK^T for 64 query rows -- two 32-row
// blocks sharing each K operand read -- and their exponentials, and hands the
// bf16 weights to wave w + 4 through LDS (double-buffered); wave w + 4 (the
// consumer) runs PV for the 64 rows, each V^T operand read serving both
// blocks.  A workgroup barrier per 32-key block.  Per iteration and pair:
// 64 rows x 32 keys x 4 x 128 FLOP, 24 KB of LDS traffic (32 KB for two
// waves of the prefill's own slot).
__global__ __launch_bounds__(512, 2) void probe_attn_pair_kernel(int iters,
                                                                 float* __restrict__ out) {
  constexpr int D = 128;
  using Lay = ChunkLayout<D>;
  __shared__ __attribute__((aligned(16))) bf16_t s0[Lay::kElemsTile];
  __shared__ __attribute__((aligned(16))) bf16_t s1[Lay::kElemsTile];
  __shared__ __attribute__((aligned(16))) u32x4 xb[2][4][64 * 4];   // [buffer][pair][lane, part]
  for (int i = threadIdx.x; i < Lay::kElemsTile; i += blockDim.x) {
    s0[i] = __builtin_bit_cast(bf16_t, (__bf16)(0.01f * (float)((i % 23) - 11)));
    s1[i] = __builtin_bit_cast(bf16_t, (__bf16)(0.01f * (float)((i % 19) - 9)));
  }
  for (int i = threadIdx.x; i < 2 * 4 * 64 * 4; i += blockDim.x)
    (&xb[0][0][0])[i] = u32x4{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
  __syncthreads();
  const int lane = threadIdx.x & 63, w = wave_id(), pair = w & 3;
  const Lay lay;
  const float c = 0.08838834764831845f * kLog2e;
  float res = 0.f;
  if (w < 4) {
    bf16x8 qf[2][8];
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) qf[r][ks] = probe_frag(lane, ks + 8 * r);
    const float nm = -0.5f;
    for (int it = 0; it < iters; ++it) {
      const bf16_t* kst = (it & 1) ? s1 : s0;
      const int H = (it >> 1) & 1;
      f32x16 s[2] = {};
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        const bf16x8 ka = *reinterpret_cast<const bf16x8*>(kst + lay.k_off(H, ks));
        s[0] = mfma32(ka, qf[0][ks], s[0]);
        s[1] = mfma32(ka, qf[1][ks], s[1]);
      }
      u32x4* dst = &xb[it & 1][pair][lane * 4];
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        bf16x8 p[2];
        res += pf_weights(s[r], c, nm, p);
        dst[2 * r] = __builtin_bit_cast(u32x4, p[0]);
        dst[2 * r + 1] = __builtin_bit_cast(u32x4, p[1]);
      }
      pf_barrier();
    }
  } else {
    f32x16 o[2][4] = {};
    for (int it = 0; it < iters; ++it) {
      const bf16_t* vst = ((it & 1) ? s0 : s1) + kPfBN * D;
      const int H = (it >> 1) & 1;
      const u32x4* src = &xb[(it + 1) & 1][pair][lane * 4];   // the previous block's weights
      bf16x8 pp[2][2];
#pragma unroll
      for (int q = 0; q < 4; ++q) pp[q >> 1][q & 1] = __builtin_bit_cast(bf16x8, src[q]);
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const int rw = 32 * H + 16 * s2;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) {
          const bf16x8 a = join_bf16x8(lds_read_tr4(vst + lay.v_off(rw, dt)),
                                       lds_read_tr4(vst + lay.v_off(rw + 8, dt)));
          o[0][dt] = mfma32(a, pp[0][s2], o[0][dt]);
          o[1][dt] = mfma32(a, pp[1][s2], o[1][dt]);
        }
      }
      pf_barrier();
    }
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int j = 0; j < 16; ++j) res += o[r][dt][j];
  }
  if (res == 1.2345e-30f) out[blockIdx.x] = res;
}

// The slot's MFMA and vector instructions in pf_full_slot's order, K and V
// operands from registers: per step one QK^T MFMA, the exponent arguments of
// the next step's scores, two exp2, the bf16 packing and row sum of the step
// before, one PV MFMA.  Two slots per iteration with the score and weight
// registers trading roles, as in the prefill loop (no copies).
struct ProbeRegs {
  bf16x8 qf[8], ka[8], va[8];
  f32x16 oacc[4];
  float l;
};

__device__ __forceinline__ void probe_reg_slot(ProbeRegs& r, const f32x16& s_cur, f32x16& s_next,
                                               bf16x8 (&p_cur)[2], const bf16x8 (&p_prev)[2],
                                               float c, float nm) {
  constexpr int kSteps = 8, kPer = 2;
#pragma unroll
  for (int i = 0; i < kSteps; ++i) asm volatile("" : "+v"(r.ka[i]), "+v"(r.va[i]));
  float x[16], w[16];
  bf16x2 pr[8];
  float sum = 0.f;
  auto arg = [&](int i) {
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
  auto pack = [&](int i) {
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
  arg(0);
  f32x16 acc = {};
#pragma unroll
  for (int i = 0; i < kSteps; ++i) {
    __builtin_amdgcn_sched_barrier(0);
    acc = mfma32(r.ka[i], r.qf[i], acc);
    if (i + 1 < kSteps) arg(i + 1);
    expo(i);
    if (i >= 1) pack(i - 1);
    r.oacc[i % 4] = mfma32(r.va[i], p_prev[i / 4], r.oacc[i % 4]);
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
  r.l += sum;
}

__global__ __launch_bounds__(512, 2) void probe_softmax_mfma_kernel(int iters,
                                                                    float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  ProbeRegs r;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    r.qf[i] = probe_frag(lane, i);
    r.ka[i] = probe_frag(lane, 11 + i);
    r.va[i] = probe_frag(lane, 29 + i);
  }
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) r.oacc[dt] = f32x16{};
  r.l = 0.f;
  f32x16 sE = {}, sO = {};
  bf16x8 pE[2] = {}, pO[2] = {};
  const float c = 0.08838834764831845f * kLog2e, nm = -0.5f;
  for (int it = 0; it < iters; ++it) {
    probe_reg_slot(r, sE, sO, pE, pO, c, nm);
    probe_reg_slot(r, sO, sE, pO, pE, c, nm);
  }
  float v = r.l;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int j = 0; j < 16; ++j) v += r.oacc[dt][j];
  if (v == 1.2345e-30f) out[blockIdx.x] = v;
}

}  // namespace
}  // namespace rag

extern "C" {

int rag_probe_page_read(const void* pool, const int32_t* page_ids, int64_t num_pages,
                        int32_t workgroups, int32_t stream_hint, void* sink,
                        hipStream_t stream) {
  if (!pool || !page_ids || !sink || num_pages < 0 || workgroups <= 0) return -1;
  if (stream_hint)
    hipLaunchKernelGGL(rag::probe_pages_kernel<true>, dim3(workgroups), dim3(256), 0, stream,
                       (const rag::u32x4*)pool, page_ids, num_pages, (uint32_t*)sink);
  else
    hipLaunchKernelGGL(rag::probe_pages_kernel<false>, dim3(workgroups), dim3(256), 0, stream,
                       (const rag::u32x4*)pool, page_ids, num_pages, (uint32_t*)sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int rag_probe_kv_page_read(const void* k_pool, const void* v_pool, const int32_t* page_ids,
                           int64_t num_pages, int32_t workgroups, int32_t pattern, void* sink,
                           hipStream_t stream) {
  if (!k_pool || !v_pool || !page_ids || !sink || num_pages < 0 || workgroups <= 0 ||
      pattern < 0 || pattern > 2)
    return -1;
  const rag::u32x4* kp = (const rag::u32x4*)k_pool;
  const rag::u32x4* vp = (const rag::u32x4*)v_pool;
  if (pattern == 0)
    hipLaunchKernelGGL((rag::probe_kv_pages_kernel<true, false>), dim3(workgroups), dim3(256),
                       0, stream, kp, vp, page_ids, num_pages, (uint32_t*)sink);
  else if (pattern == 1)
    hipLaunchKernelGGL((rag::probe_kv_pages_kernel<false, false>), dim3(workgroups), dim3(256),
                       0, stream, kp, vp, page_ids, num_pages, (uint32_t*)sink);
  else
    hipLaunchKernelGGL((rag::probe_kv_pages_kernel<false, true>), dim3(workgroups), dim3(256),
                       0, stream, kp, vp, page_ids, num_pages, (uint32_t*)sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int rag_probe_stream_read(const void* buf, int64_t bytes, int32_t workgroups,
                          int32_t stream_hint, void* sink, hipStream_t stream) {
  if (!buf || !sink || bytes < 0 || workgroups <= 0) return -1;
  if (stream_hint)
    hipLaunchKernelGGL(rag::probe_stream_kernel<true>, dim3(workgroups), dim3(256), 0, stream,
                       (const rag::u32x4*)buf, bytes / 16, (uint32_t*)sink);
  else
    hipLaunchKernelGGL(rag::probe_stream_kernel<false>, dim3(workgroups), dim3(256), 0, stream,
                       (const rag::u32x4*)buf, bytes / 16, (uint32_t*)sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int rag_probe_mfma_loop(int32_t iters, int32_t workgroups, void* sink, hipStream_t stream) {
  if (!sink || iters < 0 || workgroups <= 0) return -1;
  hipLaunchKernelGGL(rag::probe_mfma_kernel, dim3(workgroups), dim3(512), 0, stream, iters,
                     (float*)sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int rag_probe_attn_slot(int32_t iters, int32_t workgroups, void* sink, hipStream_t stream) {
  if (!sink || iters < 0 || workgroups <= 0) return -1;
  hipLaunchKernelGGL(rag::probe_attn_slot_kernel, dim3(workgroups), dim3(512), 0, stream, iters,
                     (float*)sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int rag_probe_attn_pair(int32_t iters, int32_t workgroups, void* sink, hipStream_t stream) {
  if (!sink || iters < 0 || workgroups <= 0) return -1;
  hipLaunchKernelGGL(rag::probe_attn_pair_kernel, dim3(workgroups), dim3(512), 0, stream, iters,
                     (float*)sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int rag_probe_softmax_mfma(int32_t iters, int32_t workgroups, void* sink, hipStream_t stream) {
  if (!sink || iters < 0 || workgroups <= 0) return -1;
  hipLaunchKernelGGL(rag::probe_softmax_mfma_kernel, dim3(workgroups), dim3(512), 0, stream,
                     iters, (float*)sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
