// C ABI of the group-quantized int4-weight GEMM (declared in
// include/rag_attn.h): argument validation, workspace sizing and the host-side
// weight packer.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "errors.h"
#include "awq.h"
#include "rag_attn.h"

namespace {

constexpr int32_t kGroup = 128;
constexpr int32_t kTileN = 128;
constexpr int32_t kTileM = 64;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

rag_status check_shape(const char* who, int32_t M, int32_t N, int32_t K, int32_t group_size) {
  using rag::fail;
  if (M < 0 || N <= 0 || K <= 0)
    return fail(RAG_ERR_INVALID_ARG, "%s: need M >= 0, N > 0, K > 0 (got %d, %d, %d)", who, M, N, K);
  if (group_size != kGroup)
    return fail(RAG_ERR_UNSUPPORTED, "%s: group_size must be 128 (got %d)", who, group_size);
  if (K % kGroup != 0)
    return fail(RAG_ERR_UNSUPPORTED, "%s: K must be a multiple of 128 (got %d)", who, K);
  if (N % kTileN != 0)
    return fail(RAG_ERR_UNSUPPORTED, "%s: N must be a multiple of 128 (got %d)", who, N);
  if ((M + kTileM - 1) / kTileM > 65535)
    return fail(RAG_ERR_UNSUPPORTED, "%s: M above 4,194,240 rows (got %d)", who, M);
  return RAG_OK;
}

}  // namespace

extern "C" {

size_t rag_awq_workspace_size(int32_t M, int32_t N, int32_t K, int32_t group_size) {
  if (check_shape("awq workspace", M, N, K, group_size) != RAG_OK || M == 0) return 0;
  const rag::AwqPlan p = rag::awq_plan(M, N, K);
  return p.sp_bytes + p.part_bytes + p.counter_bytes;
}

rag_status rag_awq_pack_weights(const uint8_t* q, int32_t K, int32_t N, int32_t group_size,
                                int32_t* packed) {
  using rag::fail;
  if (!q || !packed) return fail(RAG_ERR_INVALID_ARG, "awq pack: null pointer");
  if (rag_status st = check_shape("awq pack", 0, N, K, group_size); st != RAG_OK) return st;
  const int32_t groups = K / kGroup;
  for (int32_t g = 0; g < groups; ++g)
    for (int32_t n = 0; n < N; ++n)
      for (int32_t w = 0; w < 16; ++w) {
        // word 8a + 4b + c holds the 8 codes of k = 128g + 8o + j with
        // o = 4c + 2b + a, code j at bits 4(j/2) + 16(j%2)
        const int32_t o = 4 * (w & 3) + 2 * ((w >> 2) & 1) + (w >> 3);
        uint32_t word = 0;
        for (int32_t j = 0; j < 8; ++j) {
          const int64_t k = (int64_t)g * kGroup + 8 * o + j;
          const uint8_t c = q[k * N + n];
          if (c > 15)
            return fail(RAG_ERR_INVALID_ARG, "awq pack: code %u at (k=%lld, n=%d) is not 4-bit",
                        (unsigned)c, (long long)k, n);
          word |= (uint32_t)c << (4 * (j / 2) + 16 * (j % 2));
        }
        packed[((int64_t)g * N + n) * 16 + w] = (int32_t)word;
      }
  return rag::ok();
}

rag_status rag_awq_gemm(const void* x, const int32_t* qweight, const void* scales,
                        const uint8_t* zeros, void* y, int32_t M, int32_t N, int32_t K,
                        int32_t group_size, void* workspace, size_t workspace_bytes,
                        hipStream_t stream) {
  using rag::fail;
  if (!qweight || !scales || !zeros)
    return fail(RAG_ERR_INVALID_ARG, "awq gemm: null qweight/scales/zeros");
  if (rag_status st = check_shape("awq gemm", M, N, K, group_size); st != RAG_OK) return st;
  if (M == 0) return rag::ok();
  if (!x || !y) return fail(RAG_ERR_INVALID_ARG, "awq gemm: null x/y");
  if (!aligned(x, 16) || !aligned(qweight, 16) || !aligned(y, 16) || !aligned(scales, 16) ||
      !aligned(zeros, 16))
    return fail(RAG_ERR_INVALID_ARG,
                "awq gemm: x/qweight/scales/zeros/y must be 16-byte aligned");
  const size_t need = rag_awq_workspace_size(M, N, K, group_size);
  if (!workspace || workspace_bytes < need)
    return fail(RAG_ERR_WORKSPACE, "awq gemm: workspace of %zu bytes needed, %zu given", need,
                workspace ? workspace_bytes : (size_t)0);
  if (!aligned(workspace, 256))
    return fail(RAG_ERR_INVALID_ARG, "awq gemm: workspace must be 256-byte aligned");
  rag::AwqArgs a{x, qweight, scales, zeros, y, workspace, M, N, K};
  const hipError_t e = rag::launch_awq_gemm(a, stream);
  if (e != hipSuccess) return fail(RAG_ERR_HIP, "awq gemm: launch failed: %s", hipGetErrorString(e));
  return rag::ok();
}

}  // extern "C"
