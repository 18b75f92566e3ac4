// Group-quantized int4-weight x bf16-activation GEMM for gfx950: Y = X W with
// W[k, n] = (q[k, n] - z[g, n]) * s[g, n], g = k / 128 (the AWQ weight format
// of the served models, Sec. "Setup").
//
// Method.  The 4-bit codes become MFMA operands without any floating-point
// dequantization: a code q placed in the low mantissa bits of the bf16 value
// 128.0 (bits 0x4300 | q) is exactly 128 + q, so two codes become a pair of
// bf16 operands with one shift and one and-or.  Per group g the matrix cores
// accumulate P'[m, n] = sum_k X[m, k] (128 + q[k, n]) in fp32 (exact products,
// fp32 sums), and since
//     sum_k X[m, k] W[k, n] = s[g, n] * (P'[m, n] - (128 + z[g, n]) * S[g, m])
// with S[g, m] = sum of X[m, k] over the group, a short fp32 epilogue per group
// applies zero point and scale.  S comes from a small pre-pass over X.
//
// Packed weight layout (rag_awq_pack_weights): int32 [K/128][N][16].  Word
// 8h + t of column n in group g holds the codes of k = 128g + 16t + 8h + j,
// j = 0..7, code j in bits 4(j/2) + 16(j%2) .. +4.  Lane (column c, half h)
// of the MFMA B operand for k-step t then needs word 8h + t of its column: a
// lane's 8 words are 32 contiguous bytes, and the words of 32 consecutive
// columns of a group are 2 KB contiguous.
//
// Tiling: a workgroup of 4 waves computes a 64 x 128 tile of Y (wave w: all 64
// rows, columns 32w .. 32w+31, two 32x32 MFMA blocks); small batches split the
// groups over workgroups (partial sums in the workspace, reduced in fixed
// order by a second kernel, so results are deterministic).
#include "common.h"
#include "launch.h"

namespace rag {

constexpr int kAwqGroup = 128;
constexpr int kAwqBM = 64;
constexpr int kAwqBN = 128;

// S[g, m] = sum over the group of X[m, k], fp32 in k order.
__global__ __launch_bounds__(256) void awq_row_sums_kernel(const bf16_t* __restrict__ x,
                                                           float* __restrict__ s, int M, int K) {
  const int groups = K / kAwqGroup;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)groups * M) return;
  const int g = (int)(i / M), m = (int)(i % M);
  const bf16_t* row = x + (size_t)m * K + (size_t)g * kAwqGroup;
  float acc = 0.f;
#pragma unroll 4
  for (int c = 0; c < kAwqGroup / 8; ++c) {
    const bf16x8 v = as_bf16x8(load16(row + 8 * c));
#pragma unroll
    for (int e = 0; e < 8; ++e) acc += (float)v[e];
  }
  s[(size_t)g * M + m] = acc;
}

// Four bf16 pairs (128 + code) from one packed word.
__device__ __forceinline__ bf16x8 codes_to_bf16(uint32_t w) {
  u32x4 r;
  r[0] = (w & 0x000F000Fu) | 0x43004300u;
  r[1] = ((w >> 4) & 0x000F000Fu) | 0x43004300u;
  r[2] = ((w >> 8) & 0x000F000Fu) | 0x43004300u;
  r[3] = ((w >> 12) & 0x000F000Fu) | 0x43004300u;
  return as_bf16x8(r);
}

template <bool kSplit>
__global__ __launch_bounds__(256, 2) void awq_gemm_kernel(
    const bf16_t* __restrict__ x, const uint32_t* __restrict__ qw, const bf16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, const float* __restrict__ rsum, bf16_t* __restrict__ y,
    float* __restrict__ part, int M, int N, int K, int groups_per_split) {
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int l32 = lane & 31, h = lane >> 5;
  const int nt = blockIdx.x, mt = blockIdx.y, sp = blockIdx.z;
  const int m0 = mt * kAwqBM;
  const int n = nt * kAwqBN + 32 * wave + l32;     // this lane's column
  const int groups = K / kAwqGroup;
  const int g_begin = sp * groups_per_split;
  const int g_end = min(groups, g_begin + groups_per_split);

  f32x16 yacc[2];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int j = 0; j < 16; ++j) yacc[mb][j] = 0.f;
  // A-operand rows of this lane (row l32 of each 32-row block), zero past M
  const int ra0 = m0 + l32, ra1 = m0 + 32 + l32;
  const bf16_t* xa0 = x + (size_t)min(ra0, M - 1) * K + 8 * h;
  const bf16_t* xa1 = x + (size_t)min(ra1, M - 1) * K + 8 * h;
  const bool va0 = ra0 < M, va1 = ra1 < M;

  for (int g = g_begin; g < g_end; ++g) {
    const uint32_t* wp = qw + ((size_t)g * N + n) * 16 + 8 * h;
    const u32x4 w0 = *reinterpret_cast<const u32x4*>(wp);
    const u32x4 w1 = *reinterpret_cast<const u32x4*>(wp + 4);
    const float sc = (float)__builtin_bit_cast(__bf16, scales[(size_t)g * N + n]);
    const float zz = 128.f + (float)zeros[(size_t)g * N + n];
    f32x16 p0 = {}, p1 = {};
    const size_t kg = (size_t)g * kAwqGroup;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const uint32_t word = t < 4 ? w0[t] : w1[t - 4];
      const bf16x8 b = codes_to_bf16(word);
      u32x4 z4 = {0, 0, 0, 0};
      const bf16x8 a0 = as_bf16x8(va0 ? load16(xa0 + kg + 16 * t) : z4);
      const bf16x8 a1 = as_bf16x8(va1 ? load16(xa1 + kg + 16 * t) : z4);
      p0 = mfma32(a0, b, p0);
      p1 = mfma32(a1, b, p1);
    }
    // epilogue: rows 8(j/4) + 4h + j%4 of each block
    const float* sg = rsum + (size_t)g * M;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      const f32x16& p = mb ? p1 : p0;
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int r = m0 + 32 * mb + 8 * a + 4 * h;
        float sv[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) sv[b] = r + b < M ? sg[r + b] : 0.f;
#pragma unroll
        for (int b = 0; b < 4; ++b)
          yacc[mb][4 * a + b] = fmaf(sc, fmaf(-zz, sv[b], p[4 * a + b]), yacc[mb][4 * a + b]);
      }
    }
  }
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int r = m0 + 32 * mb + 8 * (j >> 2) + 4 * h + (j & 3);
      if (r >= M) continue;
      if constexpr (kSplit) {
        part[((size_t)sp * M + r) * N + n] = yacc[mb][j];
      } else {
        const __bf16 v = (__bf16)yacc[mb][j];
        y[(size_t)r * N + n] = __builtin_bit_cast(bf16_t, v);
      }
    }
}

// Y = sum of the split partials in split order, rounded to bf16.
__global__ __launch_bounds__(256) void awq_reduce_kernel(const float* __restrict__ part,
                                                         bf16_t* __restrict__ y, int64_t MN,
                                                         int splits) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= MN) return;
  float acc = 0.f;
  for (int s = 0; s < splits; ++s) acc += part[(size_t)s * MN + i];
  const __bf16 v = (__bf16)acc;
  y[i] = __builtin_bit_cast(bf16_t, v);
}

AwqPlan awq_plan(int M, int N, int K) {
  AwqPlan p;
  p.groups = K / kAwqGroup;
  p.tiles = (int64_t)((M + kAwqBM - 1) / kAwqBM) * (N / kAwqBN);
  // Fewer tiles than about two per CU: split the groups.
  int splits = 1;
  if (p.tiles > 0 && p.tiles < 512) splits = (int)std::min<int64_t>(p.groups, 512 / p.tiles);
  p.groups_per_split = (p.groups + splits - 1) / std::max(splits, 1);
  p.splits = std::max(1, (p.groups + p.groups_per_split - 1) / std::max(p.groups_per_split, 1));
  const size_t up = 255;
  p.rsum_bytes = ((size_t)p.groups * M * sizeof(float) + up) & ~up;
  p.part_bytes = p.splits > 1 ? (size_t)p.splits * M * N * sizeof(float) : 0;
  return p;
}

hipError_t launch_awq_gemm(const AwqArgs& a, hipStream_t stream) {
  const AwqPlan p = awq_plan(a.M, a.N, a.K);
  float* rsum = reinterpret_cast<float*>(a.workspace);
  float* part = reinterpret_cast<float*>(static_cast<char*>(a.workspace) + p.rsum_bytes);
  const int64_t nsum = (int64_t)p.groups * a.M;
  hipLaunchKernelGGL(awq_row_sums_kernel, dim3((unsigned)((nsum + 255) / 256)), dim3(256), 0,
                     stream, (const bf16_t*)a.x, rsum, a.M, a.K);
  const dim3 grid((unsigned)(a.N / kAwqBN), (unsigned)((a.M + kAwqBM - 1) / kAwqBM),
                  (unsigned)p.splits);
  if (p.splits > 1) {
    hipLaunchKernelGGL(awq_gemm_kernel<true>, grid, dim3(256), 0, stream, (const bf16_t*)a.x,
                       (const uint32_t*)a.qweight, (const bf16_t*)a.scales, a.zeros, rsum,
                       (bf16_t*)a.y, part, a.M, a.N, a.K, p.groups_per_split);
    const int64_t mn = (int64_t)a.M * a.N;
    hipLaunchKernelGGL(awq_reduce_kernel, dim3((unsigned)((mn + 255) / 256)), dim3(256), 0,
                       stream, part, (bf16_t*)a.y, mn, p.splits);
  } else {
    hipLaunchKernelGGL(awq_gemm_kernel<false>, grid, dim3(256), 0, stream, (const bf16_t*)a.x,
                       (const uint32_t*)a.qweight, (const bf16_t*)a.scales, a.zeros, rsum,
                       (bf16_t*)a.y, part, a.M, a.N, a.K, p.groups_per_split);
  }
  return hipGetLastError();
}

}  // namespace rag
