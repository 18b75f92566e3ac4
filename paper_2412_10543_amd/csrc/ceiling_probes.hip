// Ceiling probes for the MI355X (gfx950): what the memory system and the
// matrix cores deliver to kernels shaped like this library's, measured the
// same way (one launch, HIP events around it, by bench.py --ceilings).  They
// compute nothing of the attention method; they bound it:
//   * page reads: 4 KB pages at random places of a multi-GB pool, read with
//     16-byte loads -- the access pattern of paged decode;
//   * stream read: one large contiguous buffer, 16-byte loads;
//   * MFMA loop: v_mfma_f32_32x32x16_bf16 with independent accumulators, no
//     memory traffic -- the practical bf16 matrix rate.
// Each workgroup writes one value derived from what it read or computed, so
// nothing is optimised away.  Declared in include/ceiling_probes.h.
#include <hip/hip_runtime.h>

#include "ceiling_probes.h"
#include "common.h"

namespace rag {
namespace {

// Wave w of workgroup b reads the pages of list entries (b*4 + w)*4 .. +4,
// then the same again one grid further on; a page is 4096 bytes = 4 loads of
// 16 bytes per lane, so every wave has 16 loads (16 KB) in flight per step.
__global__ __launch_bounds__(256) void probe_pages_kernel(const u32x4* __restrict__ pool,
                                                          const int32_t* __restrict__ ids,
                                                          int64_t n_pages, uint32_t* __restrict__ out,
                                                          int stream_hint) {
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
      for (int i = 0; i < 4; ++i)
        v[j][i] = stream_hint ? __builtin_nontemporal_load(base + i * 64 + lane)
                              : base[i * 64 + lane];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc ^= v[j][i][0] ^ v[j][i][1] ^ v[j][i][2] ^ v[j][i][3];
  }
  if (acc == 0x9E3779B9u) out[blockIdx.x] = acc;   // practically never: keeps the loads
}

__global__ __launch_bounds__(256) void probe_stream_kernel(const u32x4* __restrict__ buf,
                                                           int64_t n16, uint32_t* __restrict__ out) {
  uint32_t acc = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x * 4;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x * 4 + threadIdx.x; i < n16; i += stride) {
    u32x4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      v[j] = i + j * blockDim.x < n16 ? buf[i + j * blockDim.x] : u32x4{0, 0, 0, 0};
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

}  // namespace
}  // namespace rag

extern "C" {

int rag_probe_page_read(const void* pool, const int32_t* page_ids, int64_t num_pages,
                        int32_t workgroups, int32_t stream_hint, void* sink,
                        hipStream_t stream) {
  if (!pool || !page_ids || !sink || num_pages < 0 || workgroups <= 0) return -1;
  hipLaunchKernelGGL(rag::probe_pages_kernel, dim3(workgroups), dim3(256), 0, stream,
                     (const rag::u32x4*)pool, page_ids, num_pages, (uint32_t*)sink, stream_hint);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int rag_probe_stream_read(const void* buf, int64_t bytes, int32_t workgroups, void* sink,
                          hipStream_t stream) {
  if (!buf || !sink || bytes < 0 || workgroups <= 0) return -1;
  hipLaunchKernelGGL(rag::probe_stream_kernel, dim3(workgroups), dim3(256), 0, stream,
                     (const rag::u32x4*)buf, bytes / 16, (uint32_t*)sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

int rag_probe_mfma_loop(int32_t iters, int32_t workgroups, void* sink, hipStream_t stream) {
  if (!sink || iters < 0 || workgroups <= 0) return -1;
  hipLaunchKernelGGL(rag::probe_mfma_kernel, dim3(workgroups), dim3(512), 0, stream, iters,
                     (float*)sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
