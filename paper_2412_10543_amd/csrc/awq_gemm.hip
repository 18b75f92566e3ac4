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
// Large batches: a pre-pass computes S in fp32 and stores it as three bf16
// pieces S1 + S2 + S3 = S (exact: 24 bits in 3 x 8), and the kernel folds the
// zero-point term into the matrix cores as one more MFMA per group (A = the
// pieces, B = -(128 + z), which bf16 holds exactly as bits 0xC300 | z), with a
// running rescale of the accumulators for the scale (see there).  Small
// batches need no pre-pass: the kernel stages its slice of X in LDS and forms
// S with the matrix cores (X times a ones operand), then applies zero point
// and scale with two fp32 FMAs per output element and group.
//
// Packed weight layout (rag_awq_pack_weights): int32 [K/128][N][16].  The
// 16 words of (group g, column n) are 64 contiguous bytes; word
// 8a + 4b + c holds the codes of the k-octet o = 4c + 2b + a, i.e. of
// k = 128g + 8o + j, j = 0..7, code j in bits 4(j/2) + 16(j%2) .. +4.  This
// order serves both MFMA shapes with contiguous reads: a 32x32x16 B-operand
// lane (column, half h) needs the octets 2t + h of k-steps t = 0..7, which
// are words 8h .. 8h+7 (step t at 8h + 4(t&1) + t/2); a 16x16x32 lane
// (column, quarter qq) needs the octets 4t + qq of k-steps t = 0..3, words
// 8(qq&1) + 4(qq>>1) .. +3.
#include <cstdlib>

#include "common.h"
#include "awq.h"

namespace rag {

constexpr int kAwqGroup = 128;
constexpr int kAwqCus = 256;     // MI355X compute units

// S[g, m] = sum over the group of X[m, k] (fp32), stored as bf16 pieces
// [S1, S2, S3, 0, 0, 0, 0, 0] (16 bytes per (g, m)), for the large-batch
// kernel.  16 lanes share one (g, m): lane c loads the 16-byte chunk c of the
// group's row (consecutive lanes, consecutive chunks) and the 16 partial sums
// are added with lane shuffles in a fixed order.
__global__ __launch_bounds__(256) void awq_group_sums_kernel(const bf16_t* __restrict__ x,
                                                             bf16_t* __restrict__ sp, int M,
                                                             int K) {
  const int groups = K / kAwqGroup;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t i = tid >> 4;
  const int c = threadIdx.x & 15;
  if (i >= (int64_t)groups * M) return;           // whole 16-lane groups
  const int g = (int)(i / M), m = (int)(i % M);
  const u32x4 raw = load16(x + (size_t)m * K + (size_t)g * kAwqGroup + 8 * c);
  const bf16x8 v = as_bf16x8(raw);
  float acc = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc += (float)v[e];
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) acc += __shfl_xor(acc, o, 16);
  if (c != 0) return;
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
  *reinterpret_cast<u32x4*>(sp + ((size_t)g * M + m) * 8) = out;
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
constexpr int kW = kBN * kAwqGroup / 2;          // 32768
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
  // The same copies one part at a time (parts 0-1: X rows, group sums, scales
  // and zero points; parts 2-3: code words), issued at k-steps 0-3 of the
  // previous group rather than all at once after its barrier, so that their
  // LDS writes interleave with that group's operand reads.
  auto issue_part = [&](int g, int st, int part) {
    char* S = lds + st * kStage;
    if (part < 2) {
      const bf16_t* xb = x + (size_t)m0 * K + (size_t)g * kAwqGroup;
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int j = 2 * part + jj;
        dma16_s(xb, xoff[j], (bf16_t*)(S + (4 * w + j) * 1024));
      }
      if (part == 0) {
        if (w < 2) {
          dma16_s(sp + (size_t)g * M * 8, spoff, (bf16_t*)(S + kX + kW + w * 1024));
        } else if (w == 2) {
          dma16((const char*)(scales + (size_t)g * N) + szoff, (bf16_t*)(S + kX + kW + kSP));
        } else if (w == 3) {
          if (lane < 32) dma16(zeros + (size_t)g * N + szoff, (bf16_t*)(S + kX + kW + kSP + 1024));
        }
      }
    } else {
      const uint32_t* wb = qw + ((size_t)g * N + n0) * 16;
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int j = 2 * (part - 2) + jj;
        dma16_s(wb, woff[j], (bf16_t*)(S + kX + (4 * w + j) * 1024));
      }
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
    const bool more = it + 1 < n_groups;
    const int g_next = g_begin + it + 1, st_next = (it + 1) % kStages;
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
      if (t < 4 && more) issue_part(g_next, st_next, t);
      bf16x8 anxt[4];
      if (t < 7) {
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) anxt[mb] = a_op(mb, t + 1);
      }
      bf16x8 b[2];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        b[nb] = codes_to_bf16(words[nb][t & 1][t >> 1], mask[nb], magic[nb]);
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
// Small batches (M <= 64), where streaming the codes from HBM is the cost.
// 16x16x32 MFMAs (16 rows per block: no padding rows for a decode batch of
// 16), one workgroup of W waves per 16 NB output columns (NB blocks of 16
// columns, which share each activation read) and split of the groups.  The
// waves form A column ranges of NB / A blocks (at most four: the conversion
// of the codes, about one VALU instruction per code, is what a wave's time
// goes to) by W / A group phases: wave w takes column range w % A and the
// groups [p R, p R + R) of the workgroup's G of phase p = w / A,
// R = ceil(G / (W / A)).
//
// X.  The waves of a phase first copy its groups' X (16-row blocks of 16 x 128,
// 4 KB each) into LDS with direct global -> LDS copies: each copy
// instruction moves four whole rows of a block (4 x 256 contiguous bytes, so
// no cache line is fetched twice), lane l of instruction i landing at
// position p = 64 i + l, which holds the 16-byte chunk j = (p % 16) ^ r of row
// r = p / 16.  The A operand of k-step t (lane (c, qq): row c, chunk 4 t + qq)
// is then one 16-byte LDS read at position 16 c + ((4 t + qq) ^ c): the 16
// lanes of a read group hit 16 different bank groups.  Rows past M read row
// M - 1 (their outputs are not stored).
//
// Codes.  Each wave streams its groups through a ring of register slots: the
// code words (16 contiguous bytes per lane and column block), scales and zero
// points of group i + depth, requested once group i is consumed (one row
// block) or as soon as it has taken its slot (more row blocks).
//
// Per group and 16-row block: P = sum_t X_t B_t over the 4 k-steps (B = the
// codes as bf16 128 + q), S = sum_t X_t 1 (a ones operand: lane (c, qq) gets
// the group sums of rows 4 qq .. 4 qq + 3, the rows of its outputs), and
// y += s (P - (128 + z) S) in fp32.  The sums of a column range's waves are
// added in LDS in phase (group) order.  With the groups split over
// workgroups, fp32 partials go out with
// device-coherent stores and the last workgroup of a column block to arrive
// (device-scope counter) adds them in split order and resets the counter.
// ---------------------------------------------------------------------------
namespace awq_sm {
constexpr int kXCap = 32;                        // 4 KB X blocks a workgroup can stage
constexpr int kLds = kXCap * 4096;
}  // namespace awq_sm

template <int MB, int NBW, int A, int kWaves>
__global__ __launch_bounds__(kWaves * 64) void awq_gemm_sm_kernel(
    const bf16_t* __restrict__ x, const uint32_t* __restrict__ qw,
    const bf16_t* __restrict__ scales, const uint8_t* __restrict__ zeros,
    bf16_t* __restrict__ y, float* __restrict__ part, int* __restrict__ arrivals, int M, int N,
    int K, int splits) {
  using namespace awq_sm;
  static_assert(kWaves % A == 0, "the waves split into A column ranges");
  constexpr int NB = NBW * A;                      // 16-column blocks of the workgroup
  constexpr int kPhases = kWaves / A;              // waves per column range
  constexpr int kCols = 16 * NB;
  constexpr int kThreads = kWaves * 64;
  // Ring of register slots, 8 / (MB NBW) of them, at most four (more only
  // repeat the last group's loads).  One row block: at least
  // two, each refilled once its group is consumed; larger row blocks (whose
  // groups cost more to compute than to wait for): each refilled as soon as
  // it is taken (measured, 16 / 32 / 64 rows).
  constexpr bool kLate = MB == 1;
  constexpr int kDepth0 = 8 / (MB * NBW) > 4 ? 4 : (8 / (MB * NBW) > 1 ? 8 / (MB * NBW) : 1);
  constexpr int kDepth = kLate && kDepth0 < 2 ? 2 : kDepth0;
  constexpr int kOut = MB * NBW * 4;               // accumulator values per lane
  static_assert(kWaves * kOut * 64 * 4 <= kLds, "wave sums fit the X region");
  __shared__ __attribute__((aligned(16))) char lds[kLds];
  const int lane = threadIdx.x & 63, w = wave_id();
  const int ca = w % A, ph = w / A;                // column range, group phase
  const int c = lane & 15, qq = lane >> 4;
  const int n0 = kCols * blockIdx.x + 16 * NBW * ca + c;   // columns n0 + 16 nb
  const int groups = K / kAwqGroup;
  const int spl = blockIdx.y;
  const int per_wg = (groups + splits - 1) / splits;
  const int wg_g0 = spl * per_wg;
  const int wg_end = min(groups, wg_g0 + per_wg);
  const int per_wave = (per_wg + kPhases - 1) / kPhases;
  const int g0 = wg_g0 + ph * per_wave;
  const int ng = max(0, min(per_wave, wg_end - g0));
  const uint32_t kMask = in_vgpr(0x000F000Fu), kMagic = in_vgpr(0x43004300u);
  const int wpos = 8 * (qq & 1) + 4 * (qq >> 1);   // this lane's 4 words

  // ---- X of this phase's groups into LDS, the copies dealt over the phase's
  // A waves ----
  for (int ii = ca; ii < ng * MB * 4; ii += A) {
    const int blk = (g0 - wg_g0) * MB + (ii >> 2), part4 = ii & 3;   // (group, row block)
    const int gl = blk / MB, mb = blk % MB;
    const int p = 64 * part4 + lane;
    const int r = p >> 4, j = (p & 15) ^ r;
    const int row = min(16 * mb + r, M - 1);
    dma16(x + (size_t)row * K + (size_t)(wg_g0 + gl) * kAwqGroup + 8 * j,
          (bf16_t*)(lds + blk * 4096 + part4 * 1024));
  }

  struct Slot {
    u32x4 wd[NBW];
    uint32_t sbits[NBW], z[NBW];
  };
  // everything one group needs from HBM; raw values only (arithmetic on a
  // loaded value here would wait for the load)
  auto fetch = [&](int g, Slot& sl) {
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      const size_t col = (size_t)g * N + n0 + 16 * nb;
      sl.wd[nb] = *reinterpret_cast<const u32x4*>(qw + col * 16 + wpos);
      sl.sbits[nb] = scales[col];
      sl.z[nb] = zeros[col];
    }
  };

  f32x4 yv[MB][NBW];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) yv[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  Slot ring[kDepth];
  const int g_last = g0 + max(ng, 1) - 1;
  if (ng > 0) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) fetch(min(g0 + d, g_last), ring[d]);
  }
  wait_vm<0>();                                    // this wave's X copies (and first codes) landed
  __atomic_signal_fence(__ATOMIC_SEQ_CST);         // no LDS read of X moves above the wait
  if constexpr (A > 1) __syncthreads();            // ... and those of the phase's other waves
  if (ng > 0) {
    const u32x4 ones = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};
    // Each pass takes kDepth groups, one per slot.  Refilled late (kLate),
    // there is no branch around a slot's loads, so the compiler's waits see
    // one order of requests and wait for a slot's own loads only, and the
    // refill lands in the slot's registers (no copies at the back edge,
    // which would wait for the loads just issued); passes past the wave's
    // last group recompute it and do not add it.  Refilled early, the loads
    // are unconditional too (clamped to the last group).
    for (int i0 = 0; i0 < ng; i0 += kDepth) {
#pragma unroll
      for (int d = 0; d < kDepth; ++d) {
        const int i = i0 + d;
        if constexpr (!kLate) {
          if (i >= ng) break;
        }
        const int g = min(g0 + i, g_last);
        __builtin_amdgcn_sched_barrier(0);
        const Slot sl = ring[d];
        if constexpr (!kLate) {
          fetch(min(g + kDepth, g_last), ring[d]);
          __builtin_amdgcn_sched_barrier(0);
        }
        bf16x8 xa[4][MB];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const char* blk = lds + ((g - wg_g0) * MB + mb) * 4096;
#pragma unroll
          for (int t = 0; t < 4; ++t)
            xa[t][mb] = as_bf16x8(
                *reinterpret_cast<const u32x4*>(blk + 16 * (16 * c + ((4 * t + qq) ^ c))));
        }
        f32x4 p[MB][NBW], sx[MB];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          sx[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int nb = 0; nb < NBW; ++nb) p[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          // one k-step at a time (converting every step's codes up front
          // would need their registers all at once)
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) sx[mb] = mfma16(xa[t][mb], as_bf16x8(ones), sx[mb]);
#pragma unroll
          for (int nb = 0; nb < NBW; ++nb) {
            const bf16x8 b = codes_to_bf16(sl.wd[nb][t], kMask, kMagic);
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) p[mb][nb] = mfma16(xa[t][mb], b, p[mb][nb]);
          }
        }
        if (i < ng) {
#pragma unroll
          for (int nb = 0; nb < NBW; ++nb) {
            const float sc = bf16_to_f32(sl.sbits[nb]);
            const float nz = -(float)(128 + (int)sl.z[nb]);
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
              for (int j = 0; j < 4; ++j)
                yv[mb][nb][j] = fmaf(sc, fmaf(nz, sx[mb][j], p[mb][nb][j]), yv[mb][nb][j]);
          }
        }
        if constexpr (kLate) {
          __builtin_amdgcn_sched_barrier(0);
          fetch(min(g0 + i + kDepth, g_last), ring[d]);   // slot consumed: refill it
        }
      }
    }
  }


  // ---- the waves' sums, added in wave order (the X region is free) ----
  __syncthreads();
  float* red = reinterpret_cast<float*>(lds);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
      for (int j = 0; j < 4; ++j) red[(w * kOut + (mb * NBW + nb) * 4 + j) * 64 + lane] = yv[mb][nb][j];
  __syncthreads();
  constexpr int kTot = MB * NB * 4;                // output values per lane position
  constexpr int kPer = (kTot * 64 + kThreads - 1) / kThreads;   // outputs per thread
  float tot[kPer];
  int orow[kPer], ocol[kPer];
#pragma unroll
  for (int e = 0; e < kPer; ++e) {
    const int idx = threadIdx.x + e * kThreads;     // (mb, nb, j, lane') of the tile
    const int l = idx & 63, j = (idx >> 6) & 3, nbg = (idx >> 8) % NB, mb = (idx >> 8) / NB;
    const bool have = idx < kTot * 64;
    orow[e] = have ? 16 * mb + 4 * (l >> 4) + j : M;
    ocol[e] = kCols * blockIdx.x + 16 * nbg + (l & 15);
    float acc = 0.f;
    if (have) {
      // the waves of column range nbg / NBW, in group order
      const int cw = nbg / NBW, nb = nbg % NBW;
#pragma unroll
      for (int v = 0; v < kPhases; ++v)
        acc += red[(((v * A + cw) * kOut) + (mb * NBW + nb) * 4 + j) * 64 + l];
    }
    tot[e] = acc;
  }
  if (splits == 1) {
#pragma unroll
    for (int e = 0; e < kPer; ++e)
      if (orow[e] < M) {
        const __bf16 o = (__bf16)tot[e];
        y[(size_t)orow[e] * N + ocol[e]] = __builtin_bit_cast(bf16_t, o);
      }
    return;
  }
  // ---- groups split over workgroups: fp32 partials (device-coherent stores,
  // another XCD may add them), then the last workgroup of the column block to
  // arrive adds them in split order and leaves its counter at zero ----
  __shared__ int flag;
#pragma unroll
  for (int e = 0; e < kPer; ++e)
    if (orow[e] < M) store_coherent(part + ((size_t)spl * M + orow[e]) * N + ocol[e], tot[e]);
  wait_all_memory();
  __syncthreads();
  if (threadIdx.x == 0)
    flag = __hip_atomic_fetch_add(arrivals + blockIdx.x, 1, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (flag != splits - 1) return;
  if (threadIdx.x == 0)
    __hip_atomic_store(arrivals + blockIdx.x, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // eight partials in flight at a time, added in split order
  float acc[kPer];
#pragma unroll
  for (int e = 0; e < kPer; ++e) acc[e] = 0.f;
  for (int s0 = 0; s0 < splits; s0 += 8) {
    float v[kPer][8];
#pragma unroll
    for (int e = 0; e < kPer; ++e)
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int s2 = min(s0 + u, splits - 1);
        const int row = min(orow[e], M - 1);
        v[e][u] = load_coherent(part + ((size_t)s2 * M + row) * N + ocol[e]);
      }
#pragma unroll
    for (int e = 0; e < kPer; ++e)
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (s0 + u < splits) acc[e] += v[e][u];
  }
#pragma unroll
  for (int e = 0; e < kPer; ++e) {
    if (orow[e] >= M) continue;
    const __bf16 o = (__bf16)acc[e];
    y[(size_t)orow[e] * N + ocol[e]] = __builtin_bit_cast(bf16_t, o);
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

// RAG_AWQ_SM_NB / RAG_AWQ_SM_SPLITS (read at each call) fix the small-batch
// column blocks per workgroup (2, 4 or 8, at most 8 / row blocks) and the split of the groups: a
// testing and tuning knob (any choice computes the same sums; only split
// counts change the fp32 addition order).
static int env_int(const char* name) {
  const char* e = std::getenv(name);
  return (e != nullptr && e[0] != 0) ? std::atoi(e) : 0;
}

AwqPlan awq_plan(int M, int N, int K) {
  AwqPlan p{};
  p.groups = K / kAwqGroup;
  p.large = M > 64;
  const size_t up = 255;
  p.splits = 1;
  p.groups_per_split = p.groups;
  if (p.large) {
    p.sp_bytes = ((size_t)p.groups * M * 16 + up) & ~up;
    p.tiles_m = (M + awq_lg::kBM - 1) / awq_lg::kBM;
    p.tiles_n = (N + awq_lg::kBN - 1) / awq_lg::kBN;
    p.tiles = (int64_t)p.tiles_m * p.tiles_n;
    p.tiles_per_xcd = (int)((p.tiles + kNumXcd - 1) / kNumXcd);
    // fewer tiles than CUs: split the groups (partials + a reduce pass)
    if (p.tiles < kAwqCus) {
      const int splits = (int)std::min<int64_t>(p.groups, (2 * kAwqCus) / p.tiles);
      p.groups_per_split = (p.groups + splits - 1) / splits;
      p.splits = (p.groups + p.groups_per_split - 1) / p.groups_per_split;
    }
    p.part_bytes = p.splits > 1 ? (((size_t)p.splits * M * N * sizeof(float) + up) & ~up) : 0;
    return p;
  }
  // Small batches: a workgroup stages X of at most kXCap 16-row blocks, so
  // the groups are split at least groups * MB / kXCap ways, and no further:
  // the merge of a split (coherent partial stores, arrival count, reloads)
  // costs more than the CUs a smaller grid leaves idle (the 7B o_proj at 16
  // rows: 6.5 us on 128 workgroups, 7.4 us split in two on 256).  The column
  // blocks per workgroup are the fewest (1, 2, 4, 8) for which the workgroups
  // fit one per CU (the 7B o_proj at 16 rows: 1 block, 256 workgroups, 5.0 us
  // against 6.0 us for 2 blocks on 128), else 8 (each workgroup copies X for
  // its groups: wider column tiles read it fewer times; the 7B gate_up_proj
  // at 64 rows, 47 us against 76 us with 2 blocks).
  p.tiles_m = 1;
  p.sm_mb = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  const int min_splits = (p.groups * p.sm_mb + awq_sm::kXCap - 1) / awq_sm::kXCap;
  p.sm_nb = 8;
  for (int nb : {1, 2, 4, 8}) {
    if (N % (16 * nb) != 0) continue;
    if ((int64_t)(N / (16 * nb)) * min_splits <= kAwqCus) {
      p.sm_nb = nb;
      break;
    }
  }
  if (const int nb = env_int("RAG_AWQ_SM_NB"); (nb == 1 || nb == 2 || nb == 4 || nb == 8) && N % (16 * nb) == 0)
    p.sm_nb = nb;
  p.tiles_n = N / (16 * p.sm_nb);
  // A waves share the column blocks, at most four blocks each and
  // MB * NB / A <= 8 (registers): eight blocks at 16 rows (the 7B
  // gate_up_proj) go to two waves of four, each taking a quarter of the
  // groups (14.1 us against 15.3 us for eight waves over all eight blocks;
  // two blocks per wave, 14.8 us; one, 16.2 us)
  p.sm_a = p.sm_nb / std::min({p.sm_nb, 4, 8 / p.sm_mb});
  int splits = min_splits;
  if (const int sp = env_int("RAG_AWQ_SM_SPLITS"); sp > 0) splits = std::max(min_splits, sp);
  splits = std::max(1, std::min(splits, p.groups));
  p.groups_per_split = (p.groups + splits - 1) / splits;
  p.splits = (p.groups + p.groups_per_split - 1) / p.groups_per_split;
  p.tiles = (int64_t)p.tiles_n * p.splits;
  if (p.splits > 1) {
    // arrival counters first: zero-filled once by the caller, left zero by
    // every call
    p.counter_bytes = ((size_t)p.tiles_n * sizeof(int) + up) & ~up;
    p.part_bytes = ((size_t)p.splits * M * N * sizeof(float) + up) & ~up;
  }
  return p;
}

hipError_t launch_awq_gemm(const AwqArgs& a, hipStream_t stream) {
  const AwqPlan p = awq_plan(a.M, a.N, a.K);
  char* ws = static_cast<char*>(a.workspace);
  const bf16_t* x = (const bf16_t*)a.x;
  const uint32_t* qw = (const uint32_t*)a.qweight;
  const bf16_t* sc = (const bf16_t*)a.scales;
  bf16_t* y = (bf16_t*)a.y;
  if (p.large) {
    bf16_t* sp = reinterpret_cast<bf16_t*>(ws);
    float* part = reinterpret_cast<float*>(ws + p.sp_bytes);
    const int64_t nsum = (int64_t)p.groups * a.M * 16;   // 16 lanes per row
    hipLaunchKernelGGL(awq_group_sums_kernel, dim3((unsigned)((nsum + 255) / 256)), dim3(256), 0,
                       stream, x, sp, a.M, a.K);
    const dim3 grid((unsigned)(p.tiles_per_xcd * kNumXcd), (unsigned)p.splits);
    if (p.splits > 1) {
      hipLaunchKernelGGL(awq_gemm_lg_kernel<true>, grid, dim3(awq_lg::kThreads), 0, stream, x, qw,
                         sc, a.zeros, sp, y, part, a.M, a.N, a.K, p.groups_per_split, p.tiles_m,
                         p.tiles_n, p.tiles_per_xcd);
      const int64_t mn = (int64_t)a.M * a.N;
      hipLaunchKernelGGL(awq_reduce_kernel, dim3((unsigned)((mn + 255) / 256)), dim3(256), 0,
                         stream, part, y, mn, p.splits);
    } else {
      hipLaunchKernelGGL(awq_gemm_lg_kernel<false>, grid, dim3(awq_lg::kThreads), 0, stream, x,
                         qw, sc, a.zeros, sp, y, part, a.M, a.N, a.K, p.groups_per_split,
                         p.tiles_m, p.tiles_n, p.tiles_per_xcd);
    }
    return hipGetLastError();
  }
  if ((int64_t)p.groups_per_split * p.sm_mb > awq_sm::kXCap) return hipErrorInvalidValue;
  int* counters = reinterpret_cast<int*>(ws);
  float* part = reinterpret_cast<float*>(ws + p.counter_bytes);
  const dim3 grid((unsigned)p.tiles_n, (unsigned)p.splits), block(512);
  auto go = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, grid, block, 0, stream, x, qw, sc, a.zeros, y, part, counters,
                       a.M, a.N, a.K, p.splits);
  };
  switch (p.sm_mb * 100 + p.sm_nb * 10 + p.sm_a) {
    case 121: go(awq_gemm_sm_kernel<1, 2, 1, 8>); break;
    case 111: go(awq_gemm_sm_kernel<1, 1, 1, 8>); break;
    case 211: go(awq_gemm_sm_kernel<2, 1, 1, 8>); break;
    case 411: go(awq_gemm_sm_kernel<4, 1, 1, 8>); break;
    case 141: go(awq_gemm_sm_kernel<1, 4, 1, 8>); break;
    case 182: go(awq_gemm_sm_kernel<1, 4, 2, 8>); break;
    case 221: go(awq_gemm_sm_kernel<2, 2, 1, 8>); break;
    case 241: go(awq_gemm_sm_kernel<2, 4, 1, 8>); break;
    case 282: go(awq_gemm_sm_kernel<2, 4, 2, 8>); break;
    case 421: go(awq_gemm_sm_kernel<4, 2, 1, 8>); break;
    case 442: go(awq_gemm_sm_kernel<4, 2, 2, 8>); break;
    case 484: go(awq_gemm_sm_kernel<4, 2, 4, 8>); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace rag
