// Host-side launch descriptors of the group-quantized int4-weight GEMM
// (internal; the public ABI is include/rag_attn.h).
#pragma once

#include <hip/hip_runtime.h>

#include <stddef.h>
#include <stdint.h>

namespace rag {

struct AwqArgs {
  const void* x;                // bf16 [M, K]
  const int32_t* qweight;       // packed codes [K/128][N][16]
  const void* scales;           // bf16 [K/128, N]
  const uint8_t* zeros;         // [K/128, N]
  void* y;                      // bf16 [M, N]
  void* workspace;
  int M, N, K;
};

struct AwqPlan {
  bool large;                   // M > 64: LDS-staged 128 x 512 tiles
  int groups, splits, groups_per_split;
  int tiles_m, tiles_n, tiles_per_xcd;
  int sm_mb;                    // small batches: 16-row blocks (1, 2 or 4)
  int sm_nb;                    // small batches: 16-column blocks per workgroup
  int sm_a;                     // small batches: waves across the columns (NB / A blocks each)
  int64_t tiles;
  size_t sp_bytes, part_bytes;  // large batches: group-sum pieces; split partials
  size_t counter_bytes;         // small batches split over groups: arrival counters
                                // (at the workspace's start)
};

AwqPlan awq_plan(int M, int N, int K);
hipError_t launch_awq_gemm(const AwqArgs& a, hipStream_t stream);

}  // namespace rag
