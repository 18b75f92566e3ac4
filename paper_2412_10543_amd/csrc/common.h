// Internal definitions shared by the gfx950 attention kernels and their host
// launchers.  Not part of the public ABI (include/rag_attn.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rag {

typedef uint16_t bf16_t;  // raw bf16 storage
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kNumXcd = 8;        // MI355X: 8 accelerator complex dies
constexpr float kLog2e = 1.4426950408889634f;
// Lazy rescaling: the running maximum used as the exponent reference is only
// moved when a new score exceeds it by more than 2^kRescaleLog2 in the
// exponentiated domain, so unnormalised weights stay <= 2^8 (fp32 and bf16
// hold that exactly in range).
constexpr float kRescaleLog2 = 8.0f;

// ---- MFMA wrappers (gfx950 bf16, fp32 accumulate) --------------------------
// 32x32x16: A lane l holds A[l%32][8*(l/32) .. +8], B lane l holds
// B[8*(l/32) .. +8][l%32], C lane l holds C[8*(j/4) + 4*(l/32) + j%4][l%32]
// for j = 0..15.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// 16x16x32: A lane l holds A[l%16][8*(l/16) .. +8], B lane l holds
// B[8*(l/16) .. +8][l%16], C lane l holds C[4*(l/16) + j][l%16], j = 0..3.
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ u32x4 as_u32x4(bf16x8 v) {
  return __builtin_bit_cast(u32x4, v);
}

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16x8 to_bf16x8(float a0, float a1, float a2, float a3,
                                            float a4, float a5, float a6, float a7) {
  f32x8 f = {a0, a1, a2, a3, a4, a5, a6, a7};
  return __builtin_convertvector(f, bf16x8);
}
__device__ __forceinline__ bf16x4 to_bf16x4(float a0, float a1, float a2, float a3) {
  f32x4 f = {a0, a1, a2, a3};
  return __builtin_convertvector(f, bf16x4);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float wave_xor(float x, int mask) {
  return __shfl_xor(x, mask, kWave);
}

// Index of this thread's wave in the workgroup, as a wave-uniform (scalar)
// value: everything derived from it then stays in scalar registers and
// branches on it are scalar branches, not exec-mask (divergent) ones.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
}

__device__ __forceinline__ bool wave_any(bool p) {
  return __builtin_amdgcn_ballot_w64(p) != 0;
}

// Device-coherent 4-byte store / load (global_store/load ... sc1): written
// through to, or read from, the point where all XCDs agree, with no L2
// write-back or invalidate of the whole cache.  Used only for the split-KV
// partial results that another XCD may merge.
__device__ __forceinline__ void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Waits until every memory access this wave issued has completed (the
// coherent stores above have reached the coherence point).
__device__ __forceinline__ void wait_all_memory() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Orders LDS traffic between the lanes of one wave (a wave-scope fence plus
// a scheduling barrier; no workgroup barrier is needed).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ u32x4 load16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
// 16-byte load with the non-temporal (streaming) hint: data read once.
__device__ __forceinline__ u32x4 load16_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// gfx950 transposing LDS read (ds_read_b64_tr_b16).  Within each group of 16
// lanes, lane i supplies the address of 4 consecutive bf16 values (row i of a
// 16 x 4 tile M) and receives M[i/4 + 4k][i%4] for k = 0..3.  Reading a
// row-major [key][d] tile this way yields the column (fixed d, four keys) that
// an MFMA A operand of V^T needs, with no transpose on the way into LDS.
__device__ __forceinline__ i16x4 lds_read_tr4(const bf16_t* p) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p));
}
// Direct global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4):
// lane l's 16 bytes land at lds_dst + 16*l, lds_dst being the same for the
// whole wave.  Counts as one vector-memory operation (vmcnt) and completes
// asynchronously; the caller waits on vmcnt and synchronises before reading
// the data.  Issued from inline assembly, so the compiler does not track the
// LDS write (it would otherwise make every later LDS read wait for all such
// copies whenever it cannot tell the destinations apart); M0, which holds
// the LDS address, is saved and restored around it.
__device__ __forceinline__ void dma16(const void* src, bf16_t* lds_dst) {
  typedef __attribute__((address_space(3))) char lds_char;
  const uint32_t base =
      __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_char*)lds_dst);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"                       // one wait state after writing M0
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(src), "s"(base)
      : "memory");
}

// The same copy with a wave-uniform 64-bit base in SGPRs plus a per-lane
// 32-bit byte offset (the global instruction's SADDR form): no per-lane 64-bit
// address arithmetic.  (The instruction's immediate offset would move the LDS
// destination too, so it stays 0.)
__device__ __forceinline__ void dma16_s(const void* sbase, uint32_t voff, bf16_t* lds_dst) {
  typedef __attribute__((address_space(3))) char lds_char;
  const uint32_t base =
      __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_char*)lds_dst);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(sbase), "s"(base)
      : "memory");
}

__device__ __forceinline__ bf16x8 join_bf16x8(i16x4 lo, i16x4 hi) {
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  i16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

// Workgroup index as seen by one XCD: the hardware deals consecutive
// workgroup ids round-robin to the 8 XCDs, so id n runs on XCD n % 8.  The
// returned index runs contiguously on each XCD, which keeps workgroups that
// read the same K/V rows inside one XCD's L2.
__device__ __forceinline__ void xcd_slot(int n, int& xcd, int& local) {
  xcd = n % kNumXcd;
  local = n / kNumXcd;
}

// Prefill tiling shared by host and device.  A workgroup is W waves of 32
// query rows each; the waves cover the q heads of one GQA group that read the
// same K/V (pf_heads_per_wg of them) times W / pf_heads_per_wg row blocks.
// Prefill workgroups (dense and chunked-prefill pieces) have 8 waves.
constexpr int kPfRowsPerWave = 32;
constexpr int kPfBN = 64;           // keys per K/V tile
constexpr int kPfWavesDense = 8;

__host__ __device__ constexpr int pf_heads_per_wg(int group) {
  return group % 4 == 0 ? 4 : (group % 2 == 0 ? 2 : 1);
}
__host__ __device__ constexpr int pf_rows_per_tile(int group, int waves) {
  return kPfRowsPerWave * (waves / pf_heads_per_wg(group));
}

// Decode tiling: one four-wave workgroup per (sequence, kv head, split) unit
// (eight waves inside the mixed launch), each wave two 16-token pages per
// step.
constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / kWave;
constexpr int kDecMaxGroup = 16;           // q heads per kv head (MFMA N)
constexpr int kDecMinPages = 16;           // fewest pages a balanced decode unit takes

// Per wave: the V rows of the NP pages of one step, row-major [16*NP][D + 16].
#ifndef RAG_DEC_PAGES
#define RAG_DEC_PAGES 2
#endif
constexpr int kDecPages = RAG_DEC_PAGES;   // pages per decode step
#ifndef RAG_MIXED_DEC_PAGES
#define RAG_MIXED_DEC_PAGES 2
#endif
constexpr int kMixedDecPages = RAG_MIXED_DEC_PAGES;   // the same, in the mixed launch
template <int D, int NP = kDecPages, int W = kDecWaves>
struct DecLds {
  static constexpr int kStrV = D + 16;
  static constexpr int kElemsWave = 16 * NP * kStrV;
  static constexpr int kBytes = W * kElemsWave * 2;
};

}  // namespace rag
