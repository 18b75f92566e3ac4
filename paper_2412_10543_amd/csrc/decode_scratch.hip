// Static per-device scratch for rag_attn_decode_paged_noalloc: the split-KV
// arrival counters and partial results of a decode call, for callers that
// cannot allocate device memory (code under HIP graph capture, tight serving
// loops).  The library allocates nothing for it at run time: the array below
// is part of the code object, and every GPU the library runs on holds its own
// copy until the process ends.
//
// Layout: [counters: kScratchCounters int32][partials: the rest].  The
// counter region only ever holds arrival counters.  It is zero-filled once per
// device at set-up, and every completed decode call leaves the counters it
// used at zero again (the merging workgroup resets them), so a call of any
// shape finds its counters at zero whatever ran before.  The partials need no
// clearing: every value a merge reads was written earlier in the same launch.
// Calls that overlap on one GPU share this memory and race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "errors.h"
#include "launch.h"

static constexpr size_t kScratchBytes = size_t(32) << 20;

static __device__ __align__(256) char scratch[kScratchBytes];

namespace rag {

namespace {

constexpr size_t kScratchCounters = 65536;
constexpr size_t kCounterBytes = kScratchCounters * sizeof(int);
constexpr int kMaxDevices = 64;

__global__ __launch_bounds__(256) void zero_words_kernel(int* __restrict__ p, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
}

struct DeviceScratch {
  std::once_flag once;
  hipError_t status = hipSuccess;
  char* ptr = nullptr;        // device address of this device's copy of `scratch`
};
DeviceScratch g_dev[kMaxDevices];

}  // namespace

size_t decode_scratch_capacity() { return kScratchBytes - kCounterBytes; }

rag_status decode_scratch(size_t counters, size_t partial_bytes, hipStream_t stream,
                          int** counters_out, char** partials_out) {
  if (counters > kScratchCounters)
    return fail(RAG_ERR_WORKSPACE,
                "decode (no-alloc): %zu (sequence, kv head) counters needed, the static scratch "
                "holds %zu", counters, kScratchCounters);
  if (partial_bytes > kScratchBytes - kCounterBytes)
    return fail(RAG_ERR_WORKSPACE,
                "decode (no-alloc): %zu bytes of split partials needed, the static scratch holds "
                "%zu (use rag_attn_decode_paged with a workspace, or fewer splits)",
                partial_bytes, kScratchBytes - kCounterBytes);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(RAG_ERR_HIP, "decode (no-alloc): hipGetDevice: %s",
                                   hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(RAG_ERR_UNSUPPORTED, "decode (no-alloc): device %d (at most %d devices)", dev,
                kMaxDevices);
  DeviceScratch& d = g_dev[dev];
  // Set-up, once per device with that device current: the device address of
  // its copy of the array (in host code the array's name is not a device
  // address), then the counter region zeroed by a fill kernel.
  std::call_once(d.once, [&d, stream]() {
    void* p = nullptr;
    d.status = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (d.status != hipSuccess) return;
    d.ptr = static_cast<char*>(p);
    const int n = (int)kScratchCounters;
    hipLaunchKernelGGL(zero_words_kernel, dim3((n + 255) / 256), dim3(256), 0, stream,
                       reinterpret_cast<int*>(d.ptr), n);
    d.status = hipGetLastError();
  });
  if (d.status != hipSuccess)
    return fail(RAG_ERR_HIP, "decode (no-alloc): scratch set-up: %s",
                hipGetErrorString(d.status));
  *counters_out = reinterpret_cast<int*>(d.ptr);
  *partials_out = d.ptr + kCounterBytes;
  return RAG_OK;
}

}  // namespace rag
