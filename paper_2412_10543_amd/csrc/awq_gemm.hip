// Group-quantized int4-weight x bf16-activation GEMM for gfx950: Y = X W with
// W[k, n] = (q[k, n] - z[g, n]) * s[g, n], g = k / 128 (the AWQ weight format
// of the served models, Sec. "Setup").
//
// Method.  The 4-bit codes become MFMA operands without any floating-point
// dequantization: a code q placed in the low mantissa bits of the bf16 value
// 128.0 (bits 0x4300 | q) is exactly 128 + q, so two codes become a pair of
// bf16 operands with one shift and one and-or.  For group g,
//     sum_k X[m, k] W[k, n] = s[g, n] * (P[m, n] - (128 + z[g, n]) * S[g, m]),
//     P = sum_k X[m, k] (128 + q[k, n]),   S[g, m] = sum of X[m, k] over g.
// A pre-pass computes S in fp32 and stores it as three bf16 pieces
// S1 + S2 + S3 = S (exact: 24 bits in 3 x 8).  The large-batch kernel folds
// the zero-point term into the matrix cores as a ninth MFMA per group (A =
// the pieces, B = -(128 + z), which bf16 holds exactly as bits 0xC300 | z),
// so the per-group scale is one fp32 FMA per output element.
//
// Packed weight layout (rag_awq_pack_weights): int32 [K/128][N][16].  Word
// 8h + t of column n in group g holds the codes of k = 128g + 16t + 8h + j,
// j = 0..7, code j in bits 4(j/2) + 16(j%2) .. +4.  MFMA B-operand lane
// (column c, half h) at k-step t needs word 8h + t of its column; a column's
// 16 words of one group are 64 contiguous bytes.
#include "common.h"
#include "launch.h"

namespace rag {

constexpr int kAwqGroup = 128;
constexpr int kAwqCus = 256;     // MI355X compute units

// S[g, m] = sum over the group of X[m, k] (fp32, k order), stored as bf16
// pieces [S1, S2, S3, 0, 0, 0, 0, 0] (16 bytes per (g, m)).
__global__ __launch_bounds__(256) void awq_group_sums_kernel(const bf16_t* __restrict__ x,
                                                             bf16_t* __restrict__ sp, int M,
                                                             int K) {
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
  const __bf16 s1 = (__bf16)acc;
  const float r1 = acc - (float)s1;
  const __bf16 s2 = (__bf16)r1;
  const __bf16 s3 = (__bf16)(r1 - (float)s2);
  u32x4 out;
  out[0] = (uint32_t)__builtin_bit_cast(uint16_t, s1) |
           ((uint32_t)__builtin_bit_cast(uint16_t, s2) << 16);
  out[1] = (uint32_t)__builtin_bit_cast(uint16_t, s3);
  out[2] = 0;
  out[3] = 0;
  *reinterpret_cast<u32x4*>(sp + (size_t)i * 8) = out;
}

// A value the compiler must keep in a VGPR (no constant folding).
__device__ __forceinline__ uint32_t in_vgpr(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}

// Four bf16 pairs (128 + code) from one packed word.  mask = 0x000F000F and
// magic = 0x43004300 come in registers: gfx9 VOP3 instructions take no
// literal operand, and with both constants in VGPRs each pair is one
// v_and_or_b32 (after a shift).
__device__ __forceinline__ bf16x8 codes_to_bf16(uint32_t w, uint32_t mask, uint32_t magic) {
  u32x4 r;
  r[0] = (w & mask) | magic;
  r[1] = ((w >> 4) & mask) | magic;
  r[2] = ((w >> 8) & mask) | magic;
  r[3] = ((w >> 12) & mask) | magic;
  return as_bf16x8(r);
}

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __builtin_bit_cast(float, bits16 << 16);
}

// ---------------------------------------------------------------------------
// Large batches: 8-wave workgroups (two waves per SIMD) own 128 x 512 tiles
// of Y; wave w computes all 128 rows and columns 64 w .. +64 as 4 x 2 MFMA
// blocks of 32 x 32.  Per group the workgroup stages in LDS, by direct
// global -> LDS copies issued one group ahead into a 2-stage ring:
//   X   128 rows x 128 k bf16, row r's 16-byte chunk c at position c ^ (r & 15)
//       (the MFMA A reads of 16 rows then hit 16 distinct bank groups)
//   W   512 columns x 64 bytes of codes, the 16-byte chunk j of column c at
//       position j ^ ((c >> 2) & 3) within its 1 KB copy block
//   SP  128 rows x 16 bytes of group-sum pieces
//   SZ  512 bf16 scales then 512 uint8 zero points
//
// Scale handling.  Each scale is split exactly as s = m * 2^e with |m| in
// [1, 2).  The power of two goes into the B operands: the magic constant's
// exponent field becomes 134 + e, so a code turns into (128 + q) 2^e, still
// exact in bf16 (likewise -(128 + z) 2^e for the zero-point term).  The
// accumulators hold u = y / c with c the m of the column's last group: before
// group g they are multiplied by c / m[g, n] (one fp32 multiply per element;
// the ratio lies in (1/2, 2), so u never leaves the range of y), then every
// MFMA of group g (the zero-point term and the 8 k-steps) accumulates
// straight into them, and y = u * c at the end.  There is no separate
// per-group accumulator, which is what lets a wave hold a 128 x 64 tile and
// convert each code word once for 4 row blocks.  A zero scale turns the
// column's operands to zero (mask and magic 0) and leaves c as it was.
// ---------------------------------------------------------------------------
namespace awq_lg {
constexpr int kThreads = 512;
constexpr int kBM = 128;
constexpr int kBN = 512;
constexpr int kStages = 2;
constexpr int kX = kBM * kAwqGroup * 2;          // 32768
constexpr int kW = kBN * kAwqGroup / 2;          // 16384
constexpr int kSP = kBM * 16;                    // 2048
constexpr int kSZ = kBN * 3;                     // 1536
constexpr int kStage = kX + kW + kSP + kSZ;      // 69120
constexpr int kGroupM = 8;                       // M tiles per raster group
constexpr int kOutStride = 144;                  // bytes per row of the output transpose
static_assert(kStage % 16 == 0, "stage alignment");
static_assert(8 * 64 * kOutStride <= kStages * kStage, "output transpose fits");
}  // namespace awq_lg

// vmcnt <= n (n < 64), expcnt and lgkmcnt unconstrained.
template <int n>
__device__ __forceinline__ void wait_vm() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (n & 15) | ((n >> 4) << 14));
}

// Per-column constants of one group from its bf16 scale bits: c = sign * m,
// the conversion mask and magic (exponent field 134 + e), and the bf16 bits of
// -(128 + z) 2^e.  Scales of 2^121 and above keep the excess power of two in
// c; a zero scale gives mask = magic = nz = 0 and c = 0 (the caller keeps its
// reference); inf or NaN gives c = NaN.
struct ColScale {
  float c;
  uint32_t mask, magic, nz;
};
__device__ __forceinline__ ColScale col_scale(uint32_t sb, uint32_t z) {
  const uint32_t E = (sb >> 7) & 0xFFu, mt = sb & 0x7Fu;
  int e;
  uint32_t mbits;
  if (E == 0) {                                   // bf16 subnormal: mt * 2^-133
    const int k = 31 - __builtin_clz(mt | 1u);
    mbits = (mt << (7 - k)) & 0x7Fu;
    e = k - 133;
  } else {
    mbits = mt;
    e = (int)E - 127;
  }
  const int eb = min(e, 120);
  float c = bf16_to_f32((sb & 0x8000u) | 0x3F80u | mbits);
  if (e > eb) c = ldexpf(c, e - eb);
  if (E == 0xFFu) c = __builtin_nanf("");
  const bool zero = (sb & 0x7FFFu) == 0;
  const uint32_t ex = (uint32_t)(134 + eb) << 7;
  ColScale r;
  r.c = zero ? 0.f : c;
  r.mask = zero ? 0u : 0x000F000Fu;
  r.magic = zero ? 0u : ex | (ex << 16);
  r.nz = zero ? 0u : 0x8000u | ex | z;
  return r;
}

template <bool kSplit>
__global__ __launch_bounds__(awq_lg::kThreads) void awq_gemm_lg_kernel(
    const bf16_t* __restrict__ x, const uint32_t* __restrict__ qw,
    const bf16_t* __restrict__ scales, const uint8_t* __restrict__ zeros,
    const bf16_t* __restrict__ sp, bf16_t* __restrict__ y, float* __restrict__ part, int M,
    int N, int K, int groups_per_split, int tiles_m, int tiles_n, int tiles_per_xcd) {
  using namespace awq_lg;
  __shared__ __attribute__((aligned(16))) char lds[kStages * kStage];
  const int lane = threadIdx.x & 63, w = wave_id();
  // tile: XCD-contiguous ranges of a grouped raster order (kGroupM M-tiles
  // per group, N fastest within it), so the workgroups resident on one XCD
  // share X rows and code columns in its L2
  int xcd, local;
  xcd_slot(blockIdx.x, xcd, local);
  const int pid = xcd * tiles_per_xcd + local;
  if (local >= tiles_per_xcd || pid >= tiles_m * tiles_n) return;
  const int per_group = kGroupM * tiles_n;
  const int first_m = (pid / per_group) * kGroupM;
  const int gm = min(tiles_m - first_m, kGroupM);
  const int mt = first_m + (pid % per_group) % gm;
  const int nt = (pid % per_group) / gm;
  const int m0 = mt * kBM, n0 = nt * kBN;
  const int groups = K / kAwqGroup;
  const int g_begin = blockIdx.y * groups_per_split;
  const int n_groups = min(groups, g_begin + groups_per_split) - g_begin;

  // ---- copies of one group into one stage (each wave its share) ----
  // Per-lane byte offsets do not depend on the group: computed once.
  uint32_t xoff[4], woff[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int row = 4 * (4 * w + j) + (lane >> 4);
    const int c = (lane & 15) ^ (row & 15);
    const int rr = min(m0 + row, M - 1) - m0;
    xoff[j] = (uint32_t)(rr * K * 2 + c * 16);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int cl = lane >> 2;
    const int ch = (lane & 3) ^ ((cl >> 2) & 3);
    const int col = min(16 * (4 * w + j) + cl, N - 1 - n0);
    woff[j] = (uint32_t)((col * 16 + ch * 4) * 4);
  }
  const uint32_t spoff = (uint32_t)(min(m0 + 64 * (w & 1) + lane, M - 1) * 16);
  const uint32_t szoff = w == 2 ? (uint32_t)(2 * min(n0 + 8 * lane, N - 8))
                                : (uint32_t)min(n0 + 16 * lane, N - 16);
  auto issue = [&](int g, int st) {
    char* S = lds + st * kStage;
    const bf16_t* xb = x + (size_t)m0 * K + (size_t)g * kAwqGroup;
#pragma unroll
    for (int j = 0; j < 4; ++j) dma16_s(xb, xoff[j], (bf16_t*)(S + (4 * w + j) * 1024));
    const uint32_t* wb = qw + ((size_t)g * N + n0) * 16;
#pragma unroll
    for (int j = 0; j < 4; ++j) dma16_s(wb, woff[j], (bf16_t*)(S + kX + (4 * w + j) * 1024));
    if (w < 2) {
      dma16_s(sp + (size_t)g * M * 8, spoff, (bf16_t*)(S + kX + kW + w * 1024));
    } else if (w == 2) {
      dma16((const char*)(scales + (size_t)g * N) + szoff, (bf16_t*)(S + kX + kW + kSP));
    } else if (w == 3) {
      if (lane < 32) dma16(zeros + (size_t)g * N + szoff, (bf16_t*)(S + kX + kW + kSP + 1024));
    }
  };
  const int r = lane & 31, h = lane >> 5;
  f32x16 u[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int j = 0; j < 16; ++j) u[a][b][j] = 0.f;
  float cref[2] = {1.f, 1.f};

  if (n_groups > 0) issue(g_begin, 0);
  for (int it = 0; it < n_groups; ++it) {
    // this group's copies have landed (the only ones in flight) and every
    // wave is done with the stage the next group's copies overwrite
    wait_vm<0>();
    __syncthreads();
    if (it + 1 < n_groups) issue(g_begin + it + 1, (it + 1) % kStages);
    const char* S = lds + (it % kStages) * kStage;
    const char* SX = S;
    const char* SW = S + kX;
    const char* SPc = S + kX + kW;
    const char* SZ = S + kX + kW + kSP;

    float rho[2];
    uint32_t mask[2], magic[2];
    bf16x8 bz[2];
    u32x4 words[2][2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int cl = 64 * w + 32 * nb + r;
      const ColScale cs = col_scale(*reinterpret_cast<const uint16_t*>(SZ + 2 * cl),
                                    (uint8_t)SZ[1024 + cl]);
      const bool zero = cs.mask == 0u;
      rho[nb] = zero ? 1.f : cref[nb] * __builtin_amdgcn_rcpf(cs.c);
      cref[nb] = zero ? cref[nb] : cs.c;
      mask[nb] = in_vgpr(cs.mask);
      magic[nb] = in_vgpr(cs.magic);
      u32x4 b;
      b[0] = cs.nz | (cs.nz << 16);
      b[1] = cs.nz;
      b[2] = 0;
      b[3] = 0;
      bz[nb] = as_bf16x8(b);
      const int blk = cl >> 4, ci = cl & 15;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int ch = (2 * h + q) ^ ((ci >> 2) & 3);
        words[nb][q] = *reinterpret_cast<const u32x4*>(SW + blk * 1024 + ci * 64 + ch * 16);
      }
    }
    auto a_op = [&](int mb, int t) {
      return as_bf16x8(*reinterpret_cast<const u32x4*>(
          SX + (32 * mb + r) * 256 + (((2 * t + h) ^ (r & 15)) * 16)));
    };
    bf16x8 acur[4];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) acur[mb] = a_op(mb, 0);
    // u <- u * c / m, then the group's MFMAs accumulate into u
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
      u32x4 v = *reinterpret_cast<const u32x4*>(SPc + (32 * mb + r) * 16);
      if (h) v = u32x4{0, 0, 0, 0};
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
        for (int j = 0; j < 16; ++j) u[mb][nb][j] *= rho[nb];
        u[mb][nb] = mfma32(as_bf16x8(v), bz[nb], u[mb][nb]);
      }
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      // one k-step at a time (the A operands of step t + 1 are loaded during
      // step t, no earlier: the accumulators need the registers)
      __builtin_amdgcn_sched_barrier(0);
      bf16x8 anxt[4];
      if (t < 7) {
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) anxt[mb] = a_op(mb, t + 1);
      }
      bf16x8 b[2];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        b[nb] = codes_to_bf16(words[nb][t >> 2][t & 3], mask[nb], magic[nb]);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) u[mb][nb] = mfma32(acur[mb], b[nb], u[mb][nb]);
      if (t < 7) {
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) acur[mb] = anxt[mb];
      }
    }
  }
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int j = 0; j < 16; ++j) u[mb][nb][j] *= cref[nb];

  // ---- output ----
  const bool cols_in = n0 + 64 * w < N;
  if constexpr (kSplit) {
    if (!cols_in) return;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int row = m0 + 32 * mb + 8 * (j >> 2) + 4 * h + (j & 3);
          if (row < M)
            part[((size_t)blockIdx.y * M + row) * N + n0 + 64 * w + 32 * nb + r] = u[mb][nb][j];
        }
  } else {
    // transpose through LDS so that each lane stores 16 contiguous bytes,
    // 64 rows at a time
    __syncthreads();
    char* T = lds + w * 64 * kOutStride;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
#pragma unroll
      for (int mh = 0; mh < 2; ++mh)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int row = 32 * mh + 8 * (j >> 2) + 4 * h + (j & 3);
            const __bf16 v = (__bf16)u[2 * half + mh][nb][j];
            *reinterpret_cast<__bf16*>(T + row * kOutStride + 2 * (32 * nb + r)) = v;
          }
      wave_lds_sync();
      if (cols_in) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int idx = 64 * i + lane;
          const int row = idx >> 3, ch = idx & 7;
          const int grow = m0 + 64 * half + row;
          const u32x4 v = *reinterpret_cast<const u32x4*>(T + row * kOutStride + ch * 16);
          if (grow < M)
            *reinterpret_cast<u32x4*>(y + (size_t)grow * N + n0 + 64 * w + 8 * ch) = v;
        }
      }
      wave_lds_sync();
    }
  }
}

// ---------------------------------------------------------------------------
// Small batches (M <= 64): 4-wave workgroups own 64 x 128 tiles; wave w
// computes columns 32 w .. +32 of all 64 rows, operands straight from global
// memory; the zero-point term is applied in fp32 from S = S1 + S2 + S3.
// ---------------------------------------------------------------------------
template <bool kSplit>
__global__ __launch_bounds__(256, 2) void awq_gemm_sm_kernel(
    const bf16_t* __restrict__ x, const uint32_t* __restrict__ qw, const bf16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, const bf16_t* __restrict__ sp, bf16_t* __restrict__ y,
    float* __restrict__ part, int M, int N, int K, int groups_per_split) {
  const int lane = threadIdx.x & 63, wave = wave_id();
  const int l32 = lane & 31, h = lane >> 5;
  const int nt = blockIdx.x, mt = blockIdx.y, spl = blockIdx.z;
  const int m0 = mt * 64;
  const int n = nt * 128 + 32 * wave + l32;     // this lane's column
  const int groups = K / kAwqGroup;
  const int g_begin = spl * groups_per_split;
  const int g_end = min(groups, g_begin + groups_per_split);

  f32x16 yacc[2];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int j = 0; j < 16; ++j) yacc[mb][j] = 0.f;
  const int ra0 = m0 + l32, ra1 = m0 + 32 + l32;
  const bf16_t* xa0 = x + (size_t)min(ra0, M - 1) * K + 8 * h;
  const bf16_t* xa1 = x + (size_t)min(ra1, M - 1) * K + 8 * h;
  const bool va0 = ra0 < M, va1 = ra1 < M;
  const uint32_t kMask = in_vgpr(0x000F000Fu), kMagic = in_vgpr(0x43004300u);

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
      const bf16x8 b = codes_to_bf16(word, kMask, kMagic);
      u32x4 z4 = {0, 0, 0, 0};
      const bf16x8 a0 = as_bf16x8(va0 ? load16(xa0 + kg + 16 * t) : z4);
      const bf16x8 a1 = as_bf16x8(va1 ? load16(xa1 + kg + 16 * t) : z4);
      p0 = mfma32(a0, b, p0);
      p1 = mfma32(a1, b, p1);
    }
    const bf16_t* sg = sp + (size_t)g * M * 8;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      const f32x16& pv = mb ? p1 : p0;
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int rw = m0 + 32 * mb + 8 * a + 4 * h;
        float sv[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          sv[b] = 0.f;
          if (rw + b < M) {
            const u32x2 pc = *reinterpret_cast<const u32x2*>(sg + (size_t)(rw + b) * 8);
            sv[b] = (bf16_to_f32(pc[0] & 0xFFFFu) + bf16_to_f32(pc[0] >> 16)) +
                    bf16_to_f32(pc[1] & 0xFFFFu);
          }
        }
#pragma unroll
        for (int b = 0; b < 4; ++b)
          yacc[mb][4 * a + b] = fmaf(sc, fmaf(-zz, sv[b], pv[4 * a + b]), yacc[mb][4 * a + b]);
      }
    }
  }
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int rw = m0 + 32 * mb + 8 * (j >> 2) + 4 * h + (j & 3);
      if (rw >= M) continue;
      if constexpr (kSplit) {
        part[((size_t)spl * M + rw) * N + n] = yacc[mb][j];
      } else {
        const __bf16 v = (__bf16)yacc[mb][j];
        y[(size_t)rw * N + n] = __builtin_bit_cast(bf16_t, v);
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
  AwqPlan p{};
  p.groups = K / kAwqGroup;
  p.large = M > 64;
  if (p.large) {
    p.tiles_m = (M + awq_lg::kBM - 1) / awq_lg::kBM;
    p.tiles_n = (N + awq_lg::kBN - 1) / awq_lg::kBN;
  } else {
    p.tiles_m = (M + 63) / 64;
    p.tiles_n = N / 128;
  }
  p.tiles = (int64_t)p.tiles_m * p.tiles_n;
  p.tiles_per_xcd = (int)((p.tiles + kNumXcd - 1) / kNumXcd);
  // Fewer tiles than resident workgroups: split the groups.
  const int64_t resident = p.large ? kAwqCus : 2 * kAwqCus;
  int splits = 1;
  if (p.tiles > 0 && p.tiles < resident)
    splits = (int)std::min<int64_t>(p.groups, (2 * resident) / p.tiles);
  p.groups_per_split = (p.groups + std::max(splits, 1) - 1) / std::max(splits, 1);
  p.splits = (p.groups + p.groups_per_split - 1) / p.groups_per_split;
  const size_t up = 255;
  p.sp_bytes = ((size_t)p.groups * M * 16 + up) & ~up;
  p.part_bytes = p.splits > 1 ? (size_t)p.splits * M * N * sizeof(float) : 0;
  return p;
}

hipError_t launch_awq_gemm(const AwqArgs& a, hipStream_t stream) {
  const AwqPlan p = awq_plan(a.M, a.N, a.K);
  bf16_t* sp = reinterpret_cast<bf16_t*>(a.workspace);
  float* part = reinterpret_cast<float*>(static_cast<char*>(a.workspace) + p.sp_bytes);
  const int64_t nsum = (int64_t)p.groups * a.M;
  hipLaunchKernelGGL(awq_group_sums_kernel, dim3((unsigned)((nsum + 255) / 256)), dim3(256), 0,
                     stream, (const bf16_t*)a.x, sp, a.M, a.K);
  const bf16_t* x = (const bf16_t*)a.x;
  const uint32_t* qw = (const uint32_t*)a.qweight;
  const bf16_t* sc = (const bf16_t*)a.scales;
  bf16_t* y = (bf16_t*)a.y;
  const bool split = p.splits > 1;
  if (p.large) {
    const dim3 grid((unsigned)(p.tiles_per_xcd * kNumXcd), (unsigned)p.splits);
    if (split)
      hipLaunchKernelGGL(awq_gemm_lg_kernel<true>, grid, dim3(awq_lg::kThreads), 0, stream, x, qw,
                         sc, a.zeros, sp, y, part, a.M, a.N, a.K, p.groups_per_split, p.tiles_m,
                         p.tiles_n, p.tiles_per_xcd);
    else
      hipLaunchKernelGGL(awq_gemm_lg_kernel<false>, grid, dim3(awq_lg::kThreads), 0, stream, x,
                         qw, sc, a.zeros, sp, y, part, a.M, a.N, a.K, p.groups_per_split,
                         p.tiles_m, p.tiles_n, p.tiles_per_xcd);
  } else {
    const dim3 grid((unsigned)p.tiles_n, (unsigned)p.tiles_m, (unsigned)p.splits);
    if (split)
      hipLaunchKernelGGL(awq_gemm_sm_kernel<true>, grid, dim3(256), 0, stream, x, qw, sc, a.zeros,
                         sp, y, part, a.M, a.N, a.K, p.groups_per_split);
    else
      hipLaunchKernelGGL(awq_gemm_sm_kernel<false>, grid, dim3(256), 0, stream, x, qw, sc,
                         a.zeros, sp, y, part, a.M, a.N, a.K, p.groups_per_split);
  }
  if (split) {
    const int64_t mn = (int64_t)a.M * a.N;
    hipLaunchKernelGGL(awq_reduce_kernel, dim3((unsigned)((mn + 255) / 256)), dim3(256), 0,
                       stream, part, y, mn, p.splits);
  }
  return hipGetLastError();
}

}  // namespace rag
