// Dense and dequantising GEMM with fused epilogues for gfx950 matrix cores.
//
//   y[m,n] = epi( sum_k x[m,k] * W[n,k] )   (nn.Linear convention, W is [N,K])
//
// This is the Linear block of the paper's block-level IR (Section III-A) and,
// with weight codes, its Op::DequantMatMul (Sections III-A and VI).  Mixed
// precision follows the paper's AMP policy (Section III-B): bf16 operands,
// fp32 accumulation, one rounding of the output.
//
// Design (256 threads = 4 waves in a 2x2 grid, block tile BM x BN):
//  * Both operands are K-contiguous, so every global load is a 16-byte vector
//    of one row and every stage row is 128 bytes (64 bf16 or 32 f32 of K).
//  * Dense weights (bf16 / f32): operands go global -> LDS directly
//    (global_load_lds_dwordx4, no register staging) into a ring of STAGES
//    buffers, so several K-steps are in flight at once.  At the encoder's
//    sizes a K-step holds ~0.1-0.2 us of matrix work while a memory round
//    trip costs ~0.5 us; with a single buffer in flight the kernel is
//    latency-bound.  Rows are stored unpadded with the 16-byte chunk index
//    XOR-swizzled by (row / 2) mod 8, which keeps both the DMA writes (1 KB
//    contiguous per wave) and the 16-row fragment reads conflict-free.
//  * Tiles are ordered XCD-aware: the device-side row count gives the live
//    tile count, the live tiles are spread over all 8 XCDs (workgroups are
//    dispatched round-robin over XCDs) and each XCD gets a contiguous run of
//    row tiles, so an XCD's L2 holds its own activation rows plus the weights.
//  * Quantised weights keep a register-staged double buffer (the codes are
//    converted to bf16 on their way into LDS), with 16 bytes of row padding.
//  * The MFMA computes the transposed tile: the weight rows are the A operand
//    and the activation rows the B operand, so each lane ends up owning one
//    output row m and four consecutive output columns n per register quad --
//    bias, GELU and residual are applied on those and written as 8/16-byte
//    vectors.
//  * bf16: one v_mfma_f32_32x32x16_bf16 per 16-k chunk.  fp32: eight
//    v_mfma_f32_32x32x2_f32 per 16-k chunk; lane half h takes k = h*8 + i in
//    instruction i for both operands (any consistent k order is a valid sum).
//  * int8 weights: codes are exact in bf16, so they enter the MFMA unscaled
//    and the per-channel scale multiplies the fp32 sum in the epilogue.
//  * int4 weights: one 16-byte load holds a whole group of 32 codes; each
//    (q - z) * s is formed in fp32 and rounded to bf16 on its way into LDS.
//  * Rows at or beyond M (or the device-side row count) are clamped on load
//    and skipped on store; whole blocks past the row count exit at once.
#include <algorithm>

#include "common.hpp"
#include "gemm_tile.hpp"
#include "kernels.hpp"

namespace rlx {
namespace {

// 16 int8 codes -> 16 bf16 (exact: |q| <= 127 needs 7 significand bits).
__device__ __forceinline__ void int8x16_to_bf16(uint4 src, uint4& lo, uint4& hi) {
  uint32_t w[4] = {src.x, src.y, src.z, src.w};
  uint32_t o[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float f0 = (float)(int8_t)(w[i] & 0xff);
    float f1 = (float)(int8_t)((w[i] >> 8) & 0xff);
    float f2 = (float)(int8_t)((w[i] >> 16) & 0xff);
    float f3 = (float)(int8_t)(w[i] >> 24);
    o[2 * i] = (__float_as_uint(f0) >> 16) | (__float_as_uint(f1) & 0xffff0000u);
    o[2 * i + 1] = (__float_as_uint(f2) >> 16) | (__float_as_uint(f3) & 0xffff0000u);
  }
  lo = make_uint4(o[0], o[1], o[2], o[3]);
  hi = make_uint4(o[4], o[5], o[6], o[7]);
}

// 8 int8 codes (k ascending) -> 8 bf16, exact.
__device__ __forceinline__ bf16x8_t int8x8_to_bf16(uint2 c) {
  const uint32_t w[2] = {c.x, c.y};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float f0 = (float)(int8_t)(w[i] & 0xff), f1 = (float)(int8_t)((w[i] >> 8) & 0xff);
    const float f2 = (float)(int8_t)((w[i] >> 16) & 0xff), f3 = (float)(int8_t)(w[i] >> 24);
    o[2 * i] = __builtin_amdgcn_perm(__float_as_uint(f1), __float_as_uint(f0), 0x07060302u);
    o[2 * i + 1] = __builtin_amdgcn_perm(__float_as_uint(f3), __float_as_uint(f2), 0x07060302u);
  }
  return as_bf16x8(make_uint4(o[0], o[1], o[2], o[3]));
}

// 8 int8 codes (k ascending) -> 8 bf16 of q * s, RNE.
__device__ __forceinline__ bf16x8_t int8x8_scaled_to_bf16(uint2 c, float s) {
  const uint32_t w[2] = {c.x, c.y};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    o[2 * i] = pack_bf16x2((float)(int8_t)(w[i] & 0xff) * s, (float)(int8_t)((w[i] >> 8) & 0xff) * s);
    o[2 * i + 1] = pack_bf16x2((float)(int8_t)((w[i] >> 16) & 0xff) * s, (float)(int8_t)(w[i] >> 24) * s);
  }
  return as_bf16x8(make_uint4(o[0], o[1], o[2], o[3]));
}

// 8 int4 codes (k ascending, low nibble first) -> 8 bf16 of (q - z) * s
// (Int4) or fma(q, s, m) (Int4M, z holding m), RNE: the same arithmetic as
// the whole-group conversions below.
// The low and the high nibbles go to the bytes of two words, each byte to
// fp32 with v_cvt_f32_ubyte; (q - z) * s is formed as fma(q, s, -z s), exact
// in the same way: z s (two f16 significands) needs at most 22 bits, so it is
// exact in fp32 and the fma rounds (q - z) s once, like the product of the
// exact difference.
template <Quant Q>
__device__ __forceinline__ bf16x8_t int4x8_to_bf16(uint32_t c, float s, float z) {
  const uint32_t lo = c & 0x0f0f0f0fu, hi = (c >> 4) & 0x0f0f0f0fu;
  const float zs = Q == Quant::Int4 ? -z * s : z;
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float a = (float)((lo >> (8 * j)) & 0xffu), b = (float)((hi >> (8 * j)) & 0xffu);
    o[j] = pack_bf16x2(fmaf(a, s, zs), fmaf(b, s, zs));
  }
  return as_bf16x8(make_uint4(o[0], o[1], o[2], o[3]));
}

// 16 int8 codes of one group -> 16 bf16 of q * s, RNE.
__device__ __forceinline__ void int8x16_scaled_to_bf16(uint4 src, float s, uint4& lo, uint4& hi) {
  uint32_t w[4] = {src.x, src.y, src.z, src.w};
  uint32_t o[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = pack_bf16x2((float)(int8_t)(w[i] & 0xff) * s, (float)(int8_t)((w[i] >> 8) & 0xff) * s);
    o[2 * i + 1] = pack_bf16x2((float)(int8_t)((w[i] >> 16) & 0xff) * s, (float)(int8_t)(w[i] >> 24) * s);
  }
  lo = make_uint4(o[0], o[1], o[2], o[3]);
  hi = make_uint4(o[4], o[5], o[6], o[7]);
}

// 32 packed int4 codes (one group) -> 32 bf16 of q * s + m (one fp32 rounding), RNE.
__device__ __forceinline__ void int4x32_min_to_bf16(uint4 src, float s, float m, uint4 out[4]) {
  uint32_t w[4] = {src.x, src.y, src.z, src.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t byte = (w[i] >> (8 * j)) & 0xffu;
      o[j] = pack_bf16x2(fmaf((float)(byte & 0xfu), s, m), fmaf((float)(byte >> 4), s, m));
    }
    out[i] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// 32 packed int4 codes (one group) -> 32 bf16 of (q - z) * s, RNE.
__device__ __forceinline__ void int4x32_to_bf16(uint4 src, float s, float z, uint4 out[4]) {
  uint32_t w[4] = {src.x, src.y, src.z, src.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t byte = (w[i] >> (8 * j)) & 0xffu;
      float lo = ((float)(byte & 0xfu) - z) * s;   // k = 2j   (low nibble)
      float hi = ((float)(byte >> 4) - z) * s;     // k = 2j+1 (high nibble)
      o[j] = pack_bf16x2(lo, hi);
    }
    out[i] = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

template <int BM, int BN, typename T, Quant Q, Epi E>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmParams p) {
  static_assert(BM % 64 == 0 && BN % 64 == 0, "tile");
  static_assert(Q == Quant::None || sizeof(T) == 2, "quantised weights need bf16 activations");
  constexpr int WM = BM / 2, WN = BN / 2;      // wave tile
  constexpr int TM = WM / 32, TN = WN / 32;    // 32x32 MFMA tiles per wave
  constexpr int ES = sizeof(T);
  constexpr int BK = kRowBytes / ES;           // K elements per stage (64 bf16 / 32 f32)
  constexpr int CH = BK / 16;                  // 16-k chunks per stage
  constexpr int kStage = (BM + BN) * kLdsRow;
  // weight global chunks per row per stage and LDS bytes each expands to
  constexpr int WCPR = Q == Quant::None ? 8 : (quant_int8(Q) ? 4 : 2);
  constexpr int WLDS = Q == Quant::None ? 16 : (quant_int8(Q) ? 32 : 64);
  constexpr int XLOADS = BM * 8 / kThreads;
  constexpr int WLOADS = (BN * WCPR + kThreads - 1) / kThreads;

  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * kStage];

  int M = p.M;
  if (p.m_dev) M = min(M, *p.m_dev);
  const int m0 = blockIdx.y * BM;
  const int n0 = blockIdx.x * BN;
  if (m0 >= M) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, half = lane >> 5;
  const int K = p.K;
  const int KT = K / BK;

  const uint8_t* xg = reinterpret_cast<const uint8_t*>(p.x);
  const uint8_t* wg = reinterpret_cast<const uint8_t*>(p.w);
  const size_t x_pitch = (size_t)K * ES;
  const size_t w_pitch = Q == Quant::None ? (size_t)K * ES : (quant_int8(Q) ? (size_t)K : (size_t)K / 2);
  const int wk_bytes = Q == Quant::None ? kRowBytes : (quant_int8(Q) ? 64 : 32);  // weight bytes per row per stage

  uint4 xr[XLOADS];
  uint4 wr[WLOADS];

  auto load_stage = [&](int kt) {
#pragma unroll
    for (int i = 0; i < XLOADS; ++i) {
      int idx = tid + i * kThreads;
      int r = idx >> 3, c = idx & 7;
      int row = min(m0 + r, M - 1);
      xr[i] = ld16(xg + (size_t)row * x_pitch + (size_t)kt * kRowBytes + c * 16);
    }
#pragma unroll
    for (int i = 0; i < WLOADS; ++i) {
      int idx = tid + i * kThreads;
      if (idx < BN * WCPR) {
        int r = idx / WCPR, c = idx % WCPR;
        wr[i] = ld16(wg + (size_t)(n0 + r) * w_pitch + (size_t)kt * wk_bytes + c * 16);
      }
    }
  };

  auto store_stage = [&](int kt, int buf) {
    uint8_t* xs = smem + buf * kStage;
    uint8_t* ws = xs + BM * kLdsRow;
#pragma unroll
    for (int i = 0; i < XLOADS; ++i) {
      int idx = tid + i * kThreads;
      int r = idx >> 3, c = idx & 7;
      st16(xs + r * kLdsRow + c * 16, xr[i]);
    }
#pragma unroll
    for (int i = 0; i < WLOADS; ++i) {
      int idx = tid + i * kThreads;
      if (idx < BN * WCPR) {
        int r = idx / WCPR, c = idx % WCPR;
        uint8_t* dst = ws + r * kLdsRow + c * WLDS;
        if constexpr (Q == Quant::None) {
          st16(dst, wr[i]);
        } else if constexpr (Q == Quant::Int8) {
          uint4 lo, hi;
          int8x16_to_bf16(wr[i], lo, hi);
          st16(dst, lo);
          st16(dst + 16, hi);
        } else if constexpr (Q == Quant::Int8G16) {
          const int g = kt * 4 + c;  // 16 codes per chunk, one group per chunk
          const float sg = f16_bits_to_f32(reinterpret_cast<const uint16_t*>(p.scales)[(size_t)(n0 + r) * (K / 16) + g]);
          uint4 lo, hi;
          int8x16_scaled_to_bf16(wr[i], sg, lo, hi);
          st16(dst, lo);
          st16(dst + 16, hi);
        } else if constexpr (Q == Quant::Int8G) {
          const int g = kt * 2 + (c >> 1);  // 16 codes per chunk, two chunks per group
          const float sg = f16_bits_to_f32(reinterpret_cast<const uint16_t*>(p.scales)[(size_t)(n0 + r) * (K / 32) + g]);
          uint4 lo, hi;
          int8x16_scaled_to_bf16(wr[i], sg, lo, hi);
          st16(dst, lo);
          st16(dst + 16, hi);
        } else if constexpr (Q == Quant::Int4M) {
          const size_t gi = (size_t)(n0 + r) * (K / 32) + kt * 2 + c;
          const float sg = f16_bits_to_f32(reinterpret_cast<const uint16_t*>(p.scales)[gi]);
          const float mg = f16_bits_to_f32(reinterpret_cast<const uint16_t*>(p.zeros)[gi]);
          uint4 o[4];
          int4x32_min_to_bf16(wr[i], sg, mg, o);
#pragma unroll
          for (int j = 0; j < 4; ++j) st16(dst + 16 * j, o[j]);
        } else {
          const int groups = K / 32;
          const int g = kt * 2 + c;
          const uint16_t* sc = reinterpret_cast<const uint16_t*>(p.scales);
          const uint16_t* zp = reinterpret_cast<const uint16_t*>(p.zeros);
          float s = f16_bits_to_f32(sc[(size_t)(n0 + r) * groups + g]);
          float z = f16_bits_to_f32(zp[(size_t)(n0 + r) * groups + g]);
          uint4 o[4];
          int4x32_to_bf16(wr[i], s, z, o);
#pragma unroll
          for (int j = 0; j < 4; ++j) st16(dst + 16 * j, o[j]);
        }
      }
    }
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;

  load_stage(0);
  store_stage(0, 0);
  __syncthreads();

  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) load_stage(kt + 1);
    const uint8_t* xs = smem + buf * kStage;
    const uint8_t* ws = xs + BM * kLdsRow;
#pragma unroll
    for (int q = 0; q < CH; ++q) {
      if constexpr (ES == 2) {
        bf16x8_t af[TN], bfr[TM];
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
          af[tn] = as_bf16x8(ld16(ws + (wn * WN + tn * 32 + l32) * kLdsRow + q * 32 + half * 16));
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
          bfr[tm] = as_bf16x8(ld16(xs + (wm * WM + tm * 32 + l32) * kLdsRow + q * 32 + half * 16));
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
            acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[tn], bfr[tm], acc[tm][tn], 0, 0, 0);
      } else {
        float af[TN][8], bfr[TM][8];
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          const uint8_t* src = ws + (wn * WN + tn * 32 + l32) * kLdsRow + q * 64 + half * 32;
          uint4 u0 = ld16(src), u1 = ld16(src + 16);
          af[tn][0] = __uint_as_float(u0.x); af[tn][1] = __uint_as_float(u0.y);
          af[tn][2] = __uint_as_float(u0.z); af[tn][3] = __uint_as_float(u0.w);
          af[tn][4] = __uint_as_float(u1.x); af[tn][5] = __uint_as_float(u1.y);
          af[tn][6] = __uint_as_float(u1.z); af[tn][7] = __uint_as_float(u1.w);
        }
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          const uint8_t* src = xs + (wm * WM + tm * 32 + l32) * kLdsRow + q * 64 + half * 32;
          uint4 u0 = ld16(src), u1 = ld16(src + 16);
          bfr[tm][0] = __uint_as_float(u0.x); bfr[tm][1] = __uint_as_float(u0.y);
          bfr[tm][2] = __uint_as_float(u0.z); bfr[tm][3] = __uint_as_float(u0.w);
          bfr[tm][4] = __uint_as_float(u1.x); bfr[tm][5] = __uint_as_float(u1.y);
          bfr[tm][6] = __uint_as_float(u1.z); bfr[tm][7] = __uint_as_float(u1.w);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int tm = 0; tm < TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < TN; ++tn)
              acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[tn][i], bfr[tm][i], acc[tm][tn], 0, 0, 0);
      }
    }
    if (kt + 1 < KT) store_stage(kt + 1, buf ^ 1);
    __syncthreads();
  }

  static_assert(BM * (BN * 4 + 16) <= (int)sizeof(smem), "epilogue tile fits the stage memory");
  store_tile<BM, BN, T, Q, E, TM, TN, 1>(acc, smem, p, m0, n0, M);
}

// ---------------------------------------------------------------------------
// LDS-DMA kernel for dense weights
// ---------------------------------------------------------------------------

// KS > 1 (bf16): 4*KS waves; wave group g multiplies chunks [g*CH/KS, (g+1)*CH/KS)
// of every stage into its own accumulators, summed in the epilogue.  With one
// block per CU this gives each SIMD KS waves to interleave.
//
// Quantised weights (bf16 activations, no deferred LayerNorm): the codes
// travel by DMA like dense weights and become bf16 in registers as each MFMA
// fragment is read.  int8 (per-channel or group): 64 bytes per row and stage
// at a 64-byte pitch, 16-byte chunks XOR-swizzled by (row / 4) mod 4; int4:
// 32 bytes at a 32-byte pitch, chunks swizzled by (row / 8) mod 2 -- both
// leave the fragment reads at the minimum two-way bank conflict.  Group
// scales (and zeros / mins) of the tile's rows for all of K are loaded into
// LDS once, before the first stage (gq_lds_bytes).  Each weight is formed as
// in the register-staged kernel: int8 per-channel codes exactly (scale on the
// fp32 sum in the epilogue); int8 group q s, int4 (q - z) s, int4 min
// fma(q, s, m) in fp32, rounded to bf16.
__host__ __device__ constexpr bool dma_quant_ok(Quant q) {
  return q == Quant::None || q == Quant::Int8 || q == Quant::Int8G || q == Quant::Int4 || q == Quant::Int4M ||
         q == Quant::Int8G16;
}
__host__ __device__ constexpr bool quant_grouped(Quant q) {
  return q == Quant::Int8G || q == Quant::Int4 || q == Quant::Int4M || q == Quant::Int8G16;
}
// Layouts with scales only (no zero-point / min array).
__host__ __device__ constexpr bool quant_scales_only(Quant q) { return q == Quant::Int8G || q == Quant::Int8G16; }
// LDS for the group scales (and zeros / mins) of BN rows over K.
__host__ __device__ inline int gq_lds_bytes(Quant q, int BN, int K) {
  return quant_grouped(q) ? (BN * (K / quant_group_size(q)) * 2 * (quant_scales_only(q) ? 1 : 2) + 1023) / 1024 * 1024
                          : 0;
}

// EL: the epilogue operands are requested after the first operand stage
// instead of before it (launch_dma picks it: 128-column tiles, or calls of at
// least kGemmLateEpiRows rows, where there are more tiles than CUs).
constexpr int kGemmLateEpiRows = 8192;

template <int BM, int BN, int STAGES, typename T, Epi E, int KS = 1, int LN = 0, Quant Q = Quant::None, bool EL = false>
__global__ __launch_bounds__(kThreads * KS) void gemm_dma_kernel(GemmParams p) {
  static_assert(BM % 64 == 0 && BN % 64 == 0 && STAGES >= 2 && STAGES <= 6, "tile");
  static_assert(KS == 1 || (sizeof(T) == 2 && (BK_BF16 / 16) % KS == 0), "K split over bf16 chunks");
  static_assert(dma_quant_ok(Q) && (Q == Quant::None || sizeof(T) == 2), "quantised: bf16 activations");
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int ES = sizeof(T);
  constexpr int BK = kRowBytes / ES;
  constexpr int CH = BK / 16;
  constexpr int NW = 4 * KS;            // waves
  constexpr int WB = Q == Quant::None ? kRowBytes : (quant_int8(Q) ? 64 : 32);  // weight bytes per row per stage
  constexpr int WRPK = 1024 / WB;  // weight rows per 1 KB DMA block
  constexpr int kStage = BM * kRowBytes + BN * WB;
  constexpr int XI = BM * kRowBytes / 1024;               // 1 KB DMA instructions of activations per stage
  constexpr int NI = kStage / 1024;                   // 1 KB DMA blocks per stage
  constexpr int LPS = (NI + NW - 1) / NW;             // DMA instructions per thread per stage (at most)
  static_assert(kStage % 1024 == 0, "whole 1 KB DMA blocks");
  static_assert((STAGES - 2) * LPS < 64, "vmcnt range");

  __shared__ __attribute__((aligned(1024))) uint8_t smem[STAGES * kStage];
  extern __shared__ __attribute__((aligned(1024))) uint8_t epi_lds[];  // bf16: EpiLayout (dynamic size)
  constexpr bool STAGED = ES == 2;

  int M = p.M;
  if (p.m_dev) M = min(M, *p.m_dev);
  const int n_tiles = p.N / BN;
  const int live = n_tiles * ((M + BM - 1) / BM);
  const int bid = blockIdx.x;
  if (bid >= live) return;
  // XCD-aware order: bid % 8 is the XCD; give XCD x a contiguous range of tiles.
  const int q8 = live >> 3, r8 = live & 7, xcd = bid & 7;
  const int tile = xcd * q8 + min(xcd, r8) + (bid >> 3);
  const int m0 = (tile / n_tiles) * BM;
  const int n0 = (tile % n_tiles) * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int kg = wave >> 2;  // K group (KS > 1)
  const int wm = (wave & 3) >> 1, wn = wave & 1;
  const int l32 = lane & 31, half = lane >> 5;
  const int K = p.K;
  const int KT = K / BK;
  const size_t pitch = (size_t)K * ES;

  // Per-lane sources of the DMA: instruction i of this wave fills the stage's
  // 1 KB block g = wave + i * NW.  Activation blocks (g < BM / 8) hold rows
  // 8g .. 8g+7, lane at row (lane >> 3), physical chunk (lane & 7); weight
  // blocks hold rows 8h .. +7 likewise (h = g - BM / 8), or for int8 codes
  // rows 16h .. +15 at a 64-byte pitch, lane at row (lane >> 2), chunk (lane & 3).
  // Activations are row-major, or head-major ([K/32][x_head_rows][32], 64-byte
  // rows per head) when they come from the fused attention; a 64-k stage then
  // spans two heads, and logical chunk c sits in head c/4 at dims (c%4)*8.
  const bool head_major = ES == 2 && p.x_head_rows > 0;
  const size_t x_stage = head_major ? (size_t)2 * p.x_head_rows * 64 : kRowBytes;
  const uint8_t* src[LPS];
  bool is_x[LPS];
#pragma unroll
  for (int i = 0; i < LPS; ++i) {
    const int g = min(wave + i * NW, NI - 1);  // (blocks past NI are not issued)
    is_x[i] = g < XI;
    if (g < XI) {
      const int row = 8 * g + (lane >> 3);
      const int c = swz(row, lane & 7);
      const int m = min(m0 + row, M - 1);
      src[i] = head_major ? reinterpret_cast<const uint8_t*>(p.x) + ((size_t)(c >> 2) * p.x_head_rows + m) * 64 + (c & 3) * 16
                          : reinterpret_cast<const uint8_t*>(p.x) + (size_t)m * pitch + c * 16;
    } else if constexpr (quant_int8(Q)) {
      const int row = WRPK * (g - XI) + (lane >> 2);
      const int c = (lane & 3) ^ ((row >> 2) & 3);
      src[i] = reinterpret_cast<const uint8_t*>(p.w) + (size_t)(n0 + row) * K + c * 16;
    } else if constexpr (quant_int4(Q)) {
      const int row = WRPK * (g - XI) + (lane >> 1);
      const int c = (lane & 1) ^ ((row >> 3) & 1);
      src[i] = reinterpret_cast<const uint8_t*>(p.w) + (size_t)(n0 + row) * (K / 2) + c * 16;
    } else {
      const int row = 8 * (g - XI) + (lane >> 3);
      src[i] = reinterpret_cast<const uint8_t*>(p.w) + (size_t)(n0 + row) * pitch + swz(row, lane & 7) * 16;
    }
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)smem;

  auto issue = [&](int kt, int buf) {
#pragma unroll
    for (int i = 0; i < LPS; ++i) {
      if (NI % NW != 0 && wave + i * NW >= NI) break;  // uneven split: this wave has one block fewer
      const uint32_t la = lds0 + buf * kStage + (wave + i * NW) * 1024;
      lds_dma16(src[i] + (size_t)kt * (is_x[i] ? x_stage : (size_t)WB), __builtin_amdgcn_readfirstlane(la));
    }
  };

  // Group scales (then zeros / mins) of rows n0 .. n0+BN-1, [BN][G] f16
  // each (G = K / group size), into LDS after the epilogue operands: older
  // than every stage load, so the first stage's wait covers them.
  const int G = K / quant_group_size(Q);
  uint8_t* gq = epi_lds + (STAGED ? epi_layout_of<BM, BN, E, LN>(p.K, p.N).bytes : 0);
  if constexpr (quant_grouped(Q)) {
    const int dw = BN * G / 2;  // dwords per array (G is even)
    const uint32_t gq0 = lds_addr_of(gq);
    for (int a = 0; a < (quant_scales_only(Q) ? 1 : 2); ++a) {
      const uint8_t* arr = reinterpret_cast<const uint8_t*>(a == 0 ? p.scales : p.zeros);
      for (int j = wave; j * 64 < dw; j += NW) {
        const int d = j * 64 + lane;
        if (d < dw) {
          const int row = d / (G / 2), col = d - row * (G / 2);
          lds_dma4(arr + ((size_t)(n0 + row) * G + 2 * col) * 2,
                   __builtin_amdgcn_readfirstlane(gq0 + (uint32_t)(a * dw + j * 64) * 4));
        }
      }
    }
  }
  const uint16_t* gs = reinterpret_cast<const uint16_t*>(gq);           // [BN][G] scales
  const uint16_t* gz = reinterpret_cast<const uint16_t*>(gq) + BN * G;  // [BN][G] zeros / mins

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;

  // The epilogue operands are needed only at the end.  Early (!EL): oldest in
  // every wave's memory queue, landed before the first stage is waited for.
  // Late (EL): after stage 0, so they do not delay the first stage; the first
  // wait lets this wave's epi_loads epilogue loads stay in flight, and from
  // stage 1 on they are older than the stage waited for.
  constexpr bool LATE = STAGED && EL;
  if constexpr (STAGED && !LATE) issue_epilogue_operands<BM, BN, E, LN, NW>(p, m0, n0, M, epi_lds, wave, lane);
  if (KT > 0) issue(0, 0);
  int epi_loads = 0;
  if constexpr (LATE) {
    issue_epilogue_operands<BM, BN, E, LN, NW, true>(p, m0, n0, M, epi_lds, wave, lane);
    epi_loads = epilogue_dma_count<BM, BN, E, LN, NW>(p, wave);
  }
#pragma unroll
  for (int st = 1; st < STAGES - 1; ++st)
    if (st < KT) issue(st, st);

  for (int kt0 = 0; kt0 < KT; kt0 += STAGES) {
#pragma unroll
    for (int u = 0; u < STAGES; ++u) {
      const int kt = kt0 + u;
      if (kt < KT) {
        const int extra = LATE && kt == 0 ? epi_loads : 0;
        if constexpr (LATE) {
          if (NI % NW == 0 || wave < NI % NW)
            wait_stage_plus<LPS, STAGES - 2>(min(STAGES - 2, KT - 1 - kt), extra);
          else
            wait_stage_plus<(NI % NW == 0 ? LPS : LPS - 1), STAGES - 2>(min(STAGES - 2, KT - 1 - kt), extra);
        } else {
          if (NI % NW == 0 || wave < NI % NW)
            wait_stage<LPS, STAGES - 2>(min(STAGES - 2, KT - 1 - kt));
          else
            wait_stage<(NI % NW == 0 ? LPS : LPS - 1), STAGES - 2>(min(STAGES - 2, KT - 1 - kt));
        }
        __syncthreads();  // stage kt visible to all waves; buffer of stage kt-1 is free
        const bool prefetch = kt + STAGES - 1 < KT;
        const uint8_t* xs = smem + u * kStage;
        const uint8_t* ws = xs + BM * kRowBytes;
        if constexpr (ES == 2) {
          // All of the stage's fragments are requested before the first MFMA,
          // so the LDS latency is paid once per stage.  The scheduling barrier
          // keeps the compiler from sinking each read next to its MFMA (with a
          // full wait in between), which exposes the latency once per chunk.
          constexpr int CG = CH / KS;  // chunks of this wave's K group
          bf16x8_t af[CG][TN], bfr[CG][TM];
#pragma unroll
          for (int qq = 0; qq < CG; ++qq) {
            const int q = kg * CG + qq;
#pragma unroll
            for (int tn = 0; tn < TN; ++tn) {
              const int r = wn * WN + tn * 32 + l32;
              if constexpr (quant_int8(Q)) {
                // k = 16q + 8 half .. +7: bytes 8 half.. of logical chunk q
                const uint2 c8 = *reinterpret_cast<const uint2*>(ws + r * 64 + ((q ^ ((r >> 2) & 3)) * 16) + half * 8);
                if constexpr (Q == Quant::Int8)
                  af[qq][tn] = int8x8_to_bf16(c8);
                else if constexpr (Q == Quant::Int8G16)  // one group of 16 per 16-k chunk
                  af[qq][tn] = int8x8_scaled_to_bf16(c8, f16_bits_to_f32(gs[r * G + 4 * kt + q]));
                else
                  af[qq][tn] = int8x8_scaled_to_bf16(c8, f16_bits_to_f32(gs[r * G + 2 * kt + (q >> 1)]));
              } else if constexpr (quant_int4(Q)) {
                // k = 16q + 8 half .. +7: nibbles of bytes 8q + 4 half .. +3, logical chunk q / 2
                const uint32_t c4 = *reinterpret_cast<const uint32_t*>(
                    ws + r * 32 + (((q >> 1) ^ ((r >> 3) & 1)) * 16) + (q & 1) * 8 + half * 4);
                const int gi = r * G + 2 * kt + (q >> 1);
                af[qq][tn] = int4x8_to_bf16<Q>(c4, f16_bits_to_f32(gs[gi]), f16_bits_to_f32(gz[gi]));
              } else {
                af[qq][tn] = as_bf16x8(ld16(ws + r * kRowBytes + swz(r, 2 * q + half) * 16));
              }
            }
#pragma unroll
            for (int tm = 0; tm < TM; ++tm) {
              const int r = wm * WM + tm * 32 + l32;
              bfr[qq][tm] = as_bf16x8(ld16(xs + r * kRowBytes + swz(r, 2 * q + half) * 16));
            }
          }
          // the next stage's DMA goes out after the reads: its issue can stall
          // while the memory pipeline is busy, and the reads are then in flight
          if (prefetch) issue(kt + STAGES - 1, (u + STAGES - 1) % STAGES);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int qq = 0; qq < CG; ++qq)
#pragma unroll
            for (int tm = 0; tm < TM; ++tm)
#pragma unroll
              for (int tn = 0; tn < TN; ++tn)
                acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[qq][tn], bfr[qq][tm], acc[tm][tn], 0, 0, 0);
        } else {
          if (prefetch) issue(kt + STAGES - 1, (u + STAGES - 1) % STAGES);
#pragma unroll
          for (int q = 0; q < CH; ++q) {
            float af[TN][8], bfr[TM][8];
#pragma unroll
            for (int tn = 0; tn < TN; ++tn) {
              const int r = wn * WN + tn * 32 + l32;
              const uint4 u0 = ld16(ws + r * kRowBytes + swz(r, 4 * q + 2 * half) * 16);
              const uint4 u1 = ld16(ws + r * kRowBytes + swz(r, 4 * q + 2 * half + 1) * 16);
              af[tn][0] = __uint_as_float(u0.x); af[tn][1] = __uint_as_float(u0.y);
              af[tn][2] = __uint_as_float(u0.z); af[tn][3] = __uint_as_float(u0.w);
              af[tn][4] = __uint_as_float(u1.x); af[tn][5] = __uint_as_float(u1.y);
              af[tn][6] = __uint_as_float(u1.z); af[tn][7] = __uint_as_float(u1.w);
            }
#pragma unroll
            for (int tm = 0; tm < TM; ++tm) {
              const int r = wm * WM + tm * 32 + l32;
              const uint4 u0 = ld16(xs + r * kRowBytes + swz(r, 4 * q + 2 * half) * 16);
              const uint4 u1 = ld16(xs + r * kRowBytes + swz(r, 4 * q + 2 * half + 1) * 16);
              bfr[tm][0] = __uint_as_float(u0.x); bfr[tm][1] = __uint_as_float(u0.y);
              bfr[tm][2] = __uint_as_float(u0.z); bfr[tm][3] = __uint_as_float(u0.w);
              bfr[tm][4] = __uint_as_float(u1.x); bfr[tm][5] = __uint_as_float(u1.y);
              bfr[tm][6] = __uint_as_float(u1.z); bfr[tm][7] = __uint_as_float(u1.w);
            }
#pragma unroll
            for (int i = 0; i < 8; ++i)
#pragma unroll
              for (int tm = 0; tm < TM; ++tm)
#pragma unroll
                for (int tn = 0; tn < TN; ++tn)
                  acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[tn][i], bfr[tm][i], acc[tm][tn], 0, 0, 0);
          }
        }
      }
    }
  }

  constexpr int NRB = BM * (BN * 4 + 16) <= (int)sizeof(smem) ? 1 : 2;
  static_assert(BM / NRB * (BN * 4 + 16) <= (int)sizeof(smem), "epilogue row block fits the stage memory");
  // late epilogue operands have all landed (with a single K stage the only
  // wait let them stay in flight); the epilogue's first barrier then covers
  // all waves
  if constexpr (LATE) wait_vmcnt<0>();
  store_tile<BM, BN, T, Q, E, TM, TN, NRB, KS, LN, STAGED>(acc, smem, p, m0, n0, M, epi_lds);
}

// LDS a workgroup can hold on gfx950.
constexpr size_t kMaxLdsBytes = 160 * 1024;

// Static LDS of gemm_dma_kernel<BM, BN, STAGES, T, ..., Q>: its operand ring.
template <int BM, int BN, int STAGES, typename T, Quant Q>
constexpr size_t dma_ring_bytes() {
  return (size_t)STAGES * (BM * kRowBytes + BN * (Q == Quant::None ? kRowBytes : (quant_int8(Q) ? 64 : 32)));
}

template <int BM, int BN, int STAGES, typename T, Epi E, int KS, int LN, Quant Q = Quant::None>
hipError_t launch_dma(const GemmParams& p, hipStream_t s) {
  const dim3 grid((p.N / BN) * ((p.M + BM - 1) / BM));
  const size_t epi = (sizeof(T) == 2 ? (size_t)epi_layout_of<BM, BN, E, LN>(p.K, p.N).bytes : 0) +
                     (size_t)gq_lds_bytes(Q, BN, p.K);
  // the ring (static) and the epilogue operands (dynamic) share the CU's LDS:
  // a launch asking for more than there is must never be enqueued
  if (dma_ring_bytes<BM, BN, STAGES, T, Q>() + epi > kMaxLdsBytes) return hipErrorInvalidValue;
  RLX_LOG_LAUNCH("gemm_dma_kernel", grid, dim3(kThreads * KS), epi,
                 "tile=%dx%d stages=%d %s %s ksplit=%d ln=%d epi=%s M=%d%s N=%d K=%d", BM, BN, STAGES,
                 sizeof(T) == 2 ? "bf16" : "f32", quant_name(Q), KS, LN, epi_name(E), p.M, p.m_dev ? "(device)" : "",
                 p.N, p.K);
  bool late = false;  // (only bf16 activations stage epilogue operands)
  if constexpr (sizeof(T) == 2) late = BN >= 128 || p.M >= kGemmLateEpiRows;
  if constexpr (sizeof(T) == 2) {
    if (late) {
      hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, STAGES, T, E, KS, LN, Q, true>), grid, dim3(kThreads * KS), epi, s,
                         p);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, STAGES, T, E, KS, LN, Q, false>), grid, dim3(kThreads * KS), epi, s, p);
  return hipGetLastError();
}

// Deferred-LayerNorm role bits of a call (gemm_tile.hpp).
int ln_roles(const GemmParams& p) {
  return (p.x_stats ? kLnX : 0) | (p.res_stats ? kLnRes | (p.res_scaled ? kLnResG : 0) : 0) |
         (p.y_stats ? kLnOut | (p.y_gamma ? kLnOutG : 0) : 0);
}

// Quantised weights through the DMA kernel (bf16 activations): 64 x 128 tiles
// for the wide projections, else 64 x 64.  The deferred-LayerNorm roles of
// the quantised encoder layer: the QKV and FFN-up projections read a
// gamma-scaled deferred input; the output projection and FFN-down write a
// gamma-scaled LN input, the output projection's residual being the plain
// embedding output in the first layer and a gamma-scaled one after it.
template <int BM, int BN, int STAGES, Quant Q>
hipError_t launch_dma_q_tile(const GemmParams& p, hipStream_t s) {
  constexpr int kOutG = kLnOut | kLnOutG, kResG = kLnRes | kLnResG;
  const int ln = ln_roles(p);
  switch (p.epi) {
    case Epi::None:
      if (ln == 0) return launch_dma<BM, BN, STAGES, bf16_t, Epi::None, 1, 0, Q>(p, s);
      break;
    case Epi::Bias:
      if (ln == 0) return launch_dma<BM, BN, STAGES, bf16_t, Epi::Bias, 1, 0, Q>(p, s);
      if (ln == kLnX) return launch_dma<BM, BN, STAGES, bf16_t, Epi::Bias, 1, kLnX, Q>(p, s);
      break;
    case Epi::BiasGelu:
      if (ln == 0) return launch_dma<BM, BN, STAGES, bf16_t, Epi::BiasGelu, 1, 0, Q>(p, s);
      if (ln == kLnX) return launch_dma<BM, BN, STAGES, bf16_t, Epi::BiasGelu, 1, kLnX, Q>(p, s);
      break;
    case Epi::BiasResidual:
      if (ln == 0) return launch_dma<BM, BN, STAGES, bf16_t, Epi::BiasResidual, 1, 0, Q>(p, s);
      if (ln == kOutG) return launch_dma<BM, BN, STAGES, bf16_t, Epi::BiasResidual, 1, kOutG, Q>(p, s);
      if (ln == (kResG | kOutG)) return launch_dma<BM, BN, STAGES, bf16_t, Epi::BiasResidual, 1, kResG | kOutG, Q>(p, s);
      break;
  }
  return hipErrorInvalidValue;
}

// The group scales of a tile's rows must fit the LDS next to the ring: up to
// 32 KB (for example K <= 4096 with 64 weight rows of int4 scales and zeros),
// and come by dword DMA, so 4-byte aligned; otherwise the register-staged
// kernel runs.
bool dma_q_fits(const GemmParams& p, int BN) {
  auto a4 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 3) == 0; };
  if (quant_grouped(p.quant) && (!a4(p.scales) || (!quant_scales_only(p.quant) && !a4(p.zeros)))) return false;
  return gq_lds_bytes(p.quant, BN, p.K) <= 32 * 1024;
}

template <typename T, Quant Q>
hipError_t launch_typed(const GemmParams& p, hipStream_t s);

// Measured on the quantised encoder (batch 32 x 128, per forward): the DMA
// kernel wins where K is long -- FFN-down (K = 1536) 114 -> 71 us (int8),
// 150 -> 133 us (int4) -- while at K = 384 the register-staged kernel, which
// converts each weight once per block instead of once per wave that reads
// it, is as fast for int8 and faster for int4 (FFN-up 84 vs 105 us, QKV 70
// vs 92 us).
// With a deferred LayerNorm role the DMA kernel runs at every K: its
// epilogue operands are staged in LDS, which the roles need.
template <Quant Q>
hipError_t launch_dma_q(const GemmParams& p, hipStream_t s) {
  const bool ln = ln_roles(p) != 0;
  if (p.K >= 1024 || ln) {
    if (p.N % 128 == 0 && p.N >= 1024 && dma_q_fits(p, 128)) return launch_dma_q_tile<64, 128, 4, Q>(p, s);
    if (dma_q_fits(p, 64)) return launch_dma_q_tile<64, 64, 5, Q>(p, s);
    if (ln) return hipErrorInvalidValue;
  }
  return launch_typed<bf16_t, Q>(p, s);
}

template <int BM, int BN, int STAGES, typename T, int KS = 1>
hipError_t launch_dma_tile(const GemmParams& p, hipStream_t s) {
  const int ln = ln_roles(p);  // (the gamma-scaled roles are for quantised weights: rejected here)
  if constexpr (sizeof(T) == 2) {
    // the deferred-LayerNorm combinations of the encoder layer: the QKV and
    // FFN-up projections read a deferred input; the output projection writes
    // LN1's input (its residual is the deferred layer input, or the plain
    // embedding output in the first layer); FFN-down writes LN2's input
    switch (p.epi) {
      case Epi::None:
        if (ln == 0) return launch_dma<BM, BN, STAGES, T, Epi::None, KS, 0>(p, s);
        break;
      case Epi::Bias:
        if (ln == 0) return launch_dma<BM, BN, STAGES, T, Epi::Bias, KS, 0>(p, s);
        if (ln == kLnX) return launch_dma<BM, BN, STAGES, T, Epi::Bias, KS, kLnX>(p, s);
        break;
      case Epi::BiasGelu:
        if (ln == 0) return launch_dma<BM, BN, STAGES, T, Epi::BiasGelu, KS, 0>(p, s);
        if (ln == kLnX) return launch_dma<BM, BN, STAGES, T, Epi::BiasGelu, KS, kLnX>(p, s);
        break;
      case Epi::BiasResidual:
        if (ln == 0) return launch_dma<BM, BN, STAGES, T, Epi::BiasResidual, KS, 0>(p, s);
        if (ln == kLnOut) return launch_dma<BM, BN, STAGES, T, Epi::BiasResidual, KS, kLnOut>(p, s);
        if (ln == (kLnRes | kLnOut)) return launch_dma<BM, BN, STAGES, T, Epi::BiasResidual, KS, kLnRes | kLnOut>(p, s);
        break;
    }
    return hipErrorInvalidValue;
  } else {
    if (ln != 0) return hipErrorInvalidValue;
    switch (p.epi) {
      case Epi::None: return launch_dma<BM, BN, STAGES, T, Epi::None, KS, 0>(p, s);
      case Epi::Bias: return launch_dma<BM, BN, STAGES, T, Epi::Bias, KS, 0>(p, s);
      case Epi::BiasGelu: return launch_dma<BM, BN, STAGES, T, Epi::BiasGelu, KS, 0>(p, s);
      case Epi::BiasResidual: return launch_dma<BM, BN, STAGES, T, Epi::BiasResidual, KS, 0>(p, s);
    }
    return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t launch_dense(const GemmParams& p, hipStream_t s) {
  int tile = p.tile;
  if (tile == kTileAuto) {
    // measured at the encoder's shapes (2-4 k tokens): 64x64 for N = 384, 64x128
    // for the wide projections; 128x128 only pays off from ~16 k rows up
    if (p.N % 128 == 0 && p.M >= 16384) tile = kTile128x128;
    else if (p.N % 128 == 0 && p.N >= 1024) tile = kTile64x128;
    else tile = kTile64x64;
  }
  if (p.N % 128 != 0 && (tile == kTile128x128 || tile == kTile64x128)) tile = kTile64x64;
  switch (tile) {
    // stage counts keep these configurations within 80 KB of LDS: two blocks per CU
    case kTile128x128: return launch_dma_tile<128, 128, 2, T>(p, s);
    case kTile64x128: return launch_dma_tile<64, 128, 3, T>(p, s);
    case kTile128x64: return launch_dma_tile<128, 64, 3, T>(p, s);
    // 64 x 64: one block per CU at the encoder's N = 384 shapes, so bf16 splits
    // each stage's K between two groups of four waves (eight waves per CU), and
    // the ring is four stages deep: in the forward the operands come from the
    // last-level cache or HBM, not L2, and three stages in flight measured
    // 8 us per forward faster than two
    default: return launch_dma_tile<64, 64, 4, T, sizeof(T) == 2 ? 2 : 1>(p, s);
  }
}

template <int BM, int BN, typename T, Quant Q>
hipError_t launch_tile(const GemmParams& p, hipStream_t s) {
  dim3 grid(p.N / BN, (p.M + BM - 1) / BM);
  RLX_LOG_LAUNCH("gemm_kernel", grid, dim3(kThreads), 0, "tile=%dx%d register-staged %s %s epi=%s M=%d%s N=%d K=%d",
                 BM, BN, sizeof(T) == 2 ? "bf16" : "f32", quant_name(Q), epi_name(p.epi), p.M,
                 p.m_dev ? "(device)" : "", p.N, p.K);
  switch (p.epi) {
    case Epi::None: hipLaunchKernelGGL((gemm_kernel<BM, BN, T, Q, Epi::None>), grid, dim3(kThreads), 0, s, p); break;
    case Epi::Bias: hipLaunchKernelGGL((gemm_kernel<BM, BN, T, Q, Epi::Bias>), grid, dim3(kThreads), 0, s, p); break;
    case Epi::BiasGelu:
      hipLaunchKernelGGL((gemm_kernel<BM, BN, T, Q, Epi::BiasGelu>), grid, dim3(kThreads), 0, s, p);
      break;
    case Epi::BiasResidual:
      hipLaunchKernelGGL((gemm_kernel<BM, BN, T, Q, Epi::BiasResidual>), grid, dim3(kThreads), 0, s, p);
      break;
  }
  return hipGetLastError();
}

template <typename T, Quant Q>
hipError_t launch_typed(const GemmParams& p, hipStream_t s) {
  // Pick the largest tile that still gives every CU work (256 CUs).
  const long mt128 = (p.M + 127) / 128, mt64 = (p.M + 63) / 64;
  if (p.N % 128 == 0 && mt128 * (p.N / 128) >= 256) return launch_tile<128, 128, T, Q>(p, s);
  if (p.N % 128 == 0 && mt64 * (p.N / 128) >= 256) return launch_tile<64, 128, T, Q>(p, s);
  return launch_tile<64, 64, T, Q>(p, s);
}

__global__ void dequant_unpack_kernel(const uint8_t* w, Quant q, const uint16_t* scales, const uint16_t* zeros, int N,
                                      int K, float* out) {
  const size_t total = (size_t)N * K;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const int n = (int)(i / K), k = (int)(i % K);
    if (q == Quant::Int8) {
      out[i] = (float)(int8_t)w[i] * f16_bits_to_f32(scales[n]);
    } else if (q == Quant::Int8G) {
      out[i] = (float)(int8_t)w[i] * f16_bits_to_f32(scales[(size_t)n * (K / 32) + k / 32]);
    } else if (q == Quant::Int8G16) {
      out[i] = (float)(int8_t)w[i] * f16_bits_to_f32(scales[(size_t)n * (K / 16) + k / 16]);
    } else if (q == Quant::Int4M) {
      const uint8_t byte = w[(size_t)n * (K / 2) + k / 2];
      const float code = (float)((k & 1) ? (byte >> 4) : (byte & 0xf));
      const size_t g = (size_t)n * (K / 32) + k / 32;
      out[i] = fmaf(code, f16_bits_to_f32(scales[g]), f16_bits_to_f32(zeros[g]));
    } else {
      const uint8_t byte = w[(size_t)n * (K / 2) + k / 2];
      const float code = (float)((k & 1) ? (byte >> 4) : (byte & 0xf));
      const size_t g = (size_t)n * (K / 32) + k / 32;
      out[i] = (code - f16_bits_to_f32(zeros[g])) * f16_bits_to_f32(scales[g]);
    }
  }
}

// One block per weight row n (256 threads over k).
__global__ __launch_bounds__(256) void fold_ln_weights_kernel(const bf16_t* w, int K, const float* gamma,
                                                               const float* beta, const float* bias, bf16_t* w_out,
                                                               float* u_out, float* v_out) {
  const int n = blockIdx.x, tid = threadIdx.x;
  const bf16_t* row = w + (size_t)n * K;
  bf16_t* orow = w_out + (size_t)n * K;
  double u = 0.0, v = 0.0;
  for (int k = tid; k < K; k += 256) {
    const float wk = bf16_to_f32(row[k]);
    const bf16_t f = f32_to_bf16(gamma[k] * wk);  // the product of two floats, rounded once to bf16
    orow[k] = f;
    u += (double)bf16_to_f32(f);
    v += (double)beta[k] * (double)wk;
  }
  __shared__ double red[2][4];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    u += __shfl_xor(u, o, 64);
    v += __shfl_xor(v, o, 64);
  }
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = u;
    red[1][tid >> 6] = v;
  }
  __syncthreads();
  if (tid == 0) {
    u_out[n] = (float)(red[0][0] + red[0][1] + red[0][2] + red[0][3]);
    v_out[n] = (float)(red[1][0] + red[1][1] + red[1][2] + red[1][3] + (bias ? (double)bias[n] : 0.0));
  }
}

// The fp32 dequantisation of row n, column k of quantised weights, with the
// same arithmetic as the GEMM's code conversions before their bf16 rounding:
// q * s (int8, per channel or per group), fma(q, s, -z s) = (q - z) s rounded
// once (int4 with zero points), fma(q, s, m) (int4 with mins).
__device__ __forceinline__ float deq32(const uint8_t* w, Quant q, const uint16_t* scales, const uint16_t* zeros,
                                       int n, int k, int K) {
  const int gi = n * (K / 32) + k / 32;
  if (q == Quant::Int8) return (float)(int8_t)w[(size_t)n * K + k] * f16_bits_to_f32(scales[n]);
  if (q == Quant::Int8G) return (float)(int8_t)w[(size_t)n * K + k] * f16_bits_to_f32(scales[gi]);
  if (q == Quant::Int8G16)
    return (float)(int8_t)w[(size_t)n * K + k] * f16_bits_to_f32(scales[n * (K / 16) + k / 16]);
  const uint32_t byte = w[(size_t)n * (K / 2) + k / 2];
  const float c = (float)((k & 1) ? byte >> 4 : byte & 0xfu);
  const float sc = f16_bits_to_f32(scales[gi]), z = f16_bits_to_f32(zeros[gi]);
  return q == Quant::Int4 ? fmaf(c, sc, -z * sc) : fmaf(c, sc, z);
}

// Effective weight in the dequantising GEMMs: the value the matrix cores
// multiply (q * s for int8 per channel, whose scale multiplies the fp32 sum;
// the bf16 rounding of the dequantisation otherwise).
__device__ __forceinline__ float effective_weight(const uint8_t* w, Quant q, const uint16_t* scales,
                                                  const uint16_t* zeros, int n, int k, int K) {
  const float d = deq32(w, q, scales, zeros, n, k, K);
  return q == Quant::Int8 ? d : bf16_to_f32(f32_to_bf16(d));
}

// One block per weight row n (256 threads over k).  dense_fold = false (the
// dequantising GEMMs, gamma-scaled inputs): u[n] = sum_k gamma_k W_nk over the
// effective weights.  dense_fold = true (weights dequantised to bf16 with gamma
// folded in, W'_nk = bf16(gamma_k * deq32)): u[n] = sum_k W'_nk.  Both:
// v[n] = bias[n] + sum_k beta_k W_nk.
__global__ __launch_bounds__(256) void fold_ln_quant_kernel(const uint8_t* w, Quant q, const uint16_t* scales,
                                                             const uint16_t* zeros, int K, const float* gamma,
                                                             const float* beta, const float* bias, bool dense_fold,
                                                             float* u_out, float* v_out) {
  const int n = blockIdx.x, tid = threadIdx.x;
  double u = 0.0, v = 0.0;
  for (int k = tid; k < K; k += 256) {
    if (dense_fold) {
      const float d = deq32(w, q, scales, zeros, n, k, K);
      u += (double)bf16_to_f32(f32_to_bf16(gamma[k] * d));
      v += (double)beta[k] * (double)d;
    } else {
      const double wk = effective_weight(w, q, scales, zeros, n, k, K);
      u += (double)gamma[k] * wk;
      v += (double)beta[k] * wk;
    }
  }
  __shared__ double red[2][4];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    u += __shfl_xor(u, o, 64);
    v += __shfl_xor(v, o, 64);
  }
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = u;
    red[1][tid >> 6] = v;
  }
  __syncthreads();
  if (tid == 0) {
    u_out[n] = (float)(red[0][0] + red[0][1] + red[0][2] + red[0][3]);
    v_out[n] = (float)(red[1][0] + red[1][1] + red[1][2] + red[1][3] + (bias ? (double)bias[n] : 0.0));
  }
}

// Weights of every layer to bf16 in one launch: job blockIdx.y, 16
// consecutive elements of a row per thread (a whole half group of 32), the
// same fp32 dequantisation as deq32, then bf16(gamma_k * d) for a job with a
// LayerNorm gamma to fold, else bf16(d).
__global__ __launch_bounds__(256) void dequant_jobs_kernel(const DequantJob* jobs) {
  const DequantJob& j = jobs[blockIdx.y];
  const int K = j.K;
  const int64_t e0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 16;
  if (e0 >= (int64_t)j.N * K) return;
  const int n = (int)(e0 / K), k = (int)(e0 % K);
  const Quant q = j.quant;
  const uint16_t* sc = reinterpret_cast<const uint16_t*>(j.scales);
  float d[16];
  if (quant_int8(q)) {
    const uint4 c = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint8_t*>(j.w) + (size_t)n * K + k);
    const float s = f16_bits_to_f32(q == Quant::Int8    ? sc[n]
                                    : q == Quant::Int8G ? sc[n * (K / 32) + k / 32]
                                                        : sc[n * (K / 16) + k / 16]);
    const uint32_t cw[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
    for (int i = 0; i < 16; ++i) d[i] = (float)(int8_t)((cw[i >> 2] >> (8 * (i & 3))) & 0xffu) * s;
  } else {
    const uint2 c = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint8_t*>(j.w) + (size_t)n * (K / 2) + k / 2);
    const int gi = n * (K / 32) + k / 32;
    const float s = f16_bits_to_f32(sc[gi]), z = f16_bits_to_f32(reinterpret_cast<const uint16_t*>(j.zeros)[gi]);
    const float zs = q == Quant::Int4 ? -z * s : z;
    const uint32_t cw[2] = {c.x, c.y};
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t byte = (cw[i >> 3] >> (8 * ((i >> 1) & 3))) & 0xffu;
      d[i] = fmaf((float)((i & 1) ? byte >> 4 : byte & 0xfu), s, zs);
    }
  }
  if (j.gamma) {
#pragma unroll
    for (int i = 0; i < 16; ++i) d[i] *= j.gamma[k + i];
  }
  uint32_t o[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = pack_bf16x2(d[2 * i], d[2 * i + 1]);
  uint4* dst = reinterpret_cast<uint4*>(reinterpret_cast<bf16_t*>(j.out) + e0);
  dst[0] = make_uint4(o[0], o[1], o[2], o[3]);
  dst[1] = make_uint4(o[4], o[5], o[6], o[7]);
}

}  // namespace

hipError_t launch_fold_ln_weights(const void* w, int N, int K, const float* gamma, const float* beta,
                                  const float* bias, void* w_out, float* u_out, float* v_out, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  RLX_LOG_LAUNCH("fold_ln_weights_kernel", dim3(N), dim3(256), 0, "N=%d K=%d", N, K);
  hipLaunchKernelGGL(fold_ln_weights_kernel, dim3(N), dim3(256), 0, s, reinterpret_cast<const bf16_t*>(w), K, gamma,
                     beta, bias, reinterpret_cast<bf16_t*>(w_out), u_out, v_out);
  return hipGetLastError();
}

hipError_t launch_fold_ln_quant(const void* w, Quant q, const void* scales, const void* zeros, int N, int K,
                                const float* gamma, const float* beta, const float* bias, bool dense_fold,
                                float* u_out, float* v_out, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if (!dma_quant_ok(q) || q == Quant::None || K % 32 != 0) return hipErrorInvalidValue;
  RLX_LOG_LAUNCH("fold_ln_quant_kernel", dim3(N), dim3(256), 0, "%s N=%d K=%d %s", quant_name(q), N, K,
                 dense_fold ? "bf16 fold" : "gamma-scaled inputs");
  hipLaunchKernelGGL(fold_ln_quant_kernel, dim3(N), dim3(256), 0, s, reinterpret_cast<const uint8_t*>(w), q,
                     reinterpret_cast<const uint16_t*>(scales), reinterpret_cast<const uint16_t*>(zeros), K, gamma,
                     beta, bias, dense_fold, u_out, v_out);
  return hipGetLastError();
}

hipError_t launch_dequant_jobs(const DequantJob* jobs, int njobs, int max_elems, hipStream_t s) {
  if (njobs <= 0 || max_elems <= 0) return hipSuccess;
  RLX_LOG_LAUNCH("dequant_jobs_kernel", dim3((max_elems + 4095) / 4096, njobs), dim3(256), 0,
                 "jobs=%d max N*K=%d", njobs, max_elems);
  hipLaunchKernelGGL(dequant_jobs_kernel, dim3((max_elems + 4095) / 4096, njobs), dim3(256), 0, s, jobs);
  return hipGetLastError();
}

bool gemm_deferred_ln_supported(DType dt, Quant q, int H) {
  // rows of an even number of 64-column parts (whole 16-byte statistics runs), up to 1024 columns
  return dt == DType::BF16 && (q == Quant::None || dma_quant_ok(q)) && H % 128 == 0 && H <= 64 * kLnMaxParts;
}

hipError_t launch_gemm(const GemmParams& p, hipStream_t s) {
  if (p.M <= 0) return hipSuccess;
  if (p.y_f32 && (p.dtype != DType::BF16 || p.x_stats || p.res_stats || p.y_stats)) return hipErrorInvalidValue;
  if (gemv_supported(p)) return launch_gemv(p, s);
  if ((p.x_stats && !gemm_deferred_ln_supported(p.dtype, p.quant, p.K)) ||
      ((p.res_stats || p.y_stats) && !gemm_deferred_ln_supported(p.dtype, p.quant, p.N)))
    return hipErrorInvalidValue;
  if (p.dtype == DType::F32) return launch_dense<float>(p, s);
  switch (p.quant) {
    case Quant::None: return launch_dense<bf16_t>(p, s);
    case Quant::Int8: return launch_dma_q<Quant::Int8>(p, s);
    case Quant::Int4: return launch_dma_q<Quant::Int4>(p, s);
    case Quant::Int8G: return launch_dma_q<Quant::Int8G>(p, s);
    case Quant::Int8G16: return launch_dma_q<Quant::Int8G16>(p, s);
    case Quant::Int4M: return launch_dma_q<Quant::Int4M>(p, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_dequant_unpack(const void* w, Quant q, const void* scales, const void* zeros, int N, int K,
                                 float* out, hipStream_t s) {
  const size_t total = (size_t)N * K;
  const int blocks = (int)std::min<size_t>((total + 255) / 256, 4096);
  RLX_LOG_LAUNCH("dequant_unpack_kernel", dim3(blocks), dim3(256), 0, "%s N=%d K=%d", quant_name(q), N, K);
  hipLaunchKernelGGL(dequant_unpack_kernel, dim3(blocks), dim3(256), 0, s, reinterpret_cast<const uint8_t*>(w), q,
                     reinterpret_cast<const uint16_t*>(scales), reinterpret_cast<const uint16_t*>(zeros), N, K, out);
  return hipGetLastError();
}

}  // namespace rlx
