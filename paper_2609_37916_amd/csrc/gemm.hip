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
#include "kernels.hpp"

namespace rlx {
namespace {

constexpr int kThreads = 256;
constexpr int kRowBytes = 128;            // bytes of one operand row per K stage
constexpr int kLdsRow = kRowBytes + 16;   // padded LDS row pitch in bytes
constexpr int BK_BF16 = kRowBytes / 2;   // bf16 K elements per stage

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ void st16(void* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }

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
template <Quant Q>
__device__ __forceinline__ bf16x8_t int4x8_to_bf16(uint32_t c, float s, float z) {
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float lo = (float)((c >> (8 * j)) & 0xfu), hi = (float)((c >> (8 * j + 4)) & 0xfu);
    o[j] = Q == Quant::Int4 ? pack_bf16x2((lo - z) * s, (hi - z) * s) : pack_bf16x2(fmaf(lo, s, z), fmaf(hi, s, z));
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

// 16 bytes of output: 8 bf16 or 4 f32, converted to / from fp32.
template <typename T> struct Vec16;
template <> struct Vec16<bf16_t> {
  static __device__ __forceinline__ void load(const bf16_t* p, float v[8]) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  static __device__ __forceinline__ void store(bf16_t* p, const float v[8]) {
    *reinterpret_cast<uint4*>(p) = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                              pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
  }
};
template <> struct Vec16<float> {
  static __device__ __forceinline__ void load(const float* p, float v[4]) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
  }
  static __device__ __forceinline__ void store(float* p, const float v[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
};

template <typename T> struct OutVec;
template <> struct OutVec<bf16_t> {
  static __device__ __forceinline__ void load4(const bf16_t* p, float v[4]) {
    uint2 u = *reinterpret_cast<const uint2*>(p);
    v[0] = __uint_as_float(u.x << 16); v[1] = __uint_as_float(u.x & 0xffff0000u);
    v[2] = __uint_as_float(u.y << 16); v[3] = __uint_as_float(u.y & 0xffff0000u);
  }
  static __device__ __forceinline__ void store4(bf16_t* p, const float v[4]) {
    *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
  }
};
template <> struct OutVec<float> {
  static __device__ __forceinline__ void load4(const float* p, float v[4]) {
    float4 u = *reinterpret_cast<const float4*>(p);
    v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
  }
  static __device__ __forceinline__ void store4(float* p, const float v[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
};


// Epilogue through LDS: the fp32 accumulators are written to LDS in their MFMA
// layout, then every thread takes whole 16-byte output chunks of a row, so bias,
// residual and output all move as coalesced 16-byte vectors.  (Storing straight
// from the MFMA layout spreads each wave's store over 32 rows, 16 bytes per
// row, and runs several times slower.)
// KS > 1: the block's 4*KS waves form KS groups that each accumulated a share
// of the K range for the same 64-row tile layout; the staging sums the groups'
// partials (group 0 writes, the others add in turn) before the epilogue, which
// then runs on all 256*KS threads.
// Deferred-LayerNorm roles of a dense bf16 GEMM (the GemmParams fields):
// normalise the product of a deferred input, normalise a deferred residual,
// write the partial statistics of the output.
constexpr int kLnX = 1, kLnRes = 2, kLnOut = 4;

// Epilogue operands staged in LDS (dense bf16 kernels): the block's per-column
// vectors [bias, fold_u, res_gamma, res_beta][BN] (f32), its residual tile
// [BM][BN] (bf16) and the partial statistics of its rows ([BM][K/64] for x,
// [BM][N/64] for the residual).  Every region is a whole number of 1 KB DMA
// blocks.  They are requested before the first operand stage, so by the
// epilogue they have long landed and the epilogue reads no global memory.
// Each statistics region has 128 bytes of slack (a row's merge reads
// kLnMaxParts entries), and is followed by the rows' merged (mean, rstd)
// ([2][BM] float2: x, residual), which the epilogue forms once per row.
struct EpiLayout {
  int res_off, xst_off, rst_off, mrg_off, bytes;
};
__host__ __device__ inline EpiLayout epi_layout(int BM, int BN, bool res, bool xst, bool rst, int K, int N) {
  EpiLayout L;
  int off = 16 * BN;  // four f32 vectors of BN
  L.res_off = off;
  if (res) off += BM * BN * 2;
  L.xst_off = off;
  if (xst) off += (BM * (K / 64) * 8 + 128 + 1023) / 1024 * 1024;
  L.rst_off = off;
  if (rst) off += (BM * (N / 64) * 8 + 128 + 1023) / 1024 * 1024;
  L.mrg_off = off;
  if (xst || rst) off += (2 * BM * 8 + 1023) / 1024 * 1024;
  L.bytes = off;
  return L;
}
template <int BM, int BN, Epi E, int LN>
__host__ __device__ inline EpiLayout epi_layout_of(int K, int N) {
  return epi_layout(BM, BN, E == Epi::BiasResidual, (LN & kLnX) != 0, (LN & kLnRes) != 0, K, N);
}

// Merges the partial statistics staged at `epi` into each row's (mean, rstd)
// at the EpiLayout's mrg region: x rows at [0, BM), residual rows at [BM, 2BM).
// One thread per row.
template <int BM, int BN, Epi E, int LN>
__device__ __forceinline__ void merge_row_stats(const GemmParams& p, uint8_t* epi, int tid) {
  if constexpr ((LN & (kLnX | kLnRes)) != 0) {
    const EpiLayout lay = epi_layout_of<BM, BN, E, LN>(p.K, p.N);
    float2* mrg = reinterpret_cast<float2*>(epi + lay.mrg_off);
    if (tid < BM) {
      if constexpr ((LN & kLnX) != 0)
        mrg[tid] = merge_ln_lds(reinterpret_cast<const float2*>(epi + lay.xst_off) + tid * (p.K >> 6), p.K >> 6,
                                p.ln_eps);
      if constexpr ((LN & kLnRes) != 0)
        mrg[BM + tid] = merge_ln_lds(reinterpret_cast<const float2*>(epi + lay.rst_off) + tid * (p.N >> 6),
                                     p.N >> 6, p.ln_eps);
    }
  }
}

// STAGED: the epilogue operands come from LDS at `epi` (EpiLayout), else from
// global memory (no deferred LayerNorm then).
template <int BM, int BN, typename T, Quant Q, Epi E, int TM, int TN, int NRB, int KS = 1, int LN = 0,
          bool STAGED = false>
__device__ __forceinline__ void store_tile(const f32x16_t (&acc)[TM][TN], uint8_t* lds, const GemmParams& p, int m0,
                                           int n0, int M, uint8_t* epi = nullptr) {
  static_assert(NRB == 1 || NRB == 2, "row blocks follow the 2 wave rows");
  static_assert(LN == 0 || (sizeof(T) == 2 && Q == Quant::None && STAGED), "deferred LayerNorm: dense bf16");
  static_assert(!STAGED || sizeof(T) == 2, "staged epilogue operands: bf16");
  static_assert(!(LN & kLnRes) || E == Epi::BiasResidual, "a deferred residual needs the residual epilogue");
  static_assert(KS == 1 || NRB == 1, "split-K tiles stage all rows at once");
  static_assert(kThreads * KS >= BM, "one thread per row merges the row statistics");
  constexpr int NT = kThreads * KS;
  constexpr int ES = sizeof(T);
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int PITCH = BN * 4 + 16;  // bytes; 16 rows of a column land on distinct banks
  constexpr int EPC = 16 / (int)sizeof(T);
  constexpr int CPR = BN / EPC;
  constexpr int RB = BM / NRB;        // rows staged at a time
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kg = wave >> 2;  // K group
  const int wm = (wave & 3) >> 1, wn = wave & 1, l32 = lane & 31, half = lane >> 5;
  const int N = p.N;
  T* y = reinterpret_cast<T*>(p.y);
  const T* res = reinterpret_cast<const T*>(p.residual);
  const uint16_t* qs = reinterpret_cast<const uint16_t*>(p.scales);
  const EpiLayout lay = epi_layout_of<BM, BN, E, LN>(p.K, N);
  const float* vec = reinterpret_cast<const float*>(epi);  // [4][BN]: bias, fold_u, res_gamma, res_beta
  float2* mrg = reinterpret_cast<float2*>(epi + lay.mrg_off);  // [2][BM]: (mean, rstd) of x rows, residual rows
  // one thread per row merges the rows' statistics while the others stage
  // their accumulators; the barrier after the staging publishes them
  merge_row_stats<BM, BN, E, LN>(p, epi, tid);
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    __syncthreads();  // the operand stages (or the previous row block) are no longer read
#pragma unroll
    for (int g = 0; g < KS; ++g) {
      if (g > 0) __syncthreads();  // the previous group's partial is in place
      if (kg == g && (NRB == 1 || wm == rb)) {
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int r = wm * WM + tm * 32 + l32 - rb * RB;
              const int c = wn * WN + tn * 32 + 8 * i + 4 * half;
              float4* dst = reinterpret_cast<float4*>(lds + r * PITCH + c * 4);
              float4 v = make_float4(acc[tm][tn][4 * i], acc[tm][tn][4 * i + 1], acc[tm][tn][4 * i + 2],
                                     acc[tm][tn][4 * i + 3]);
              if (g > 0) {
                const float4 o = *dst;
                v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
              }
              *dst = v;
            }
      }
    }
    __syncthreads();
    // compile-time trip count: the bias and residual loads of all of a
    // thread's chunks are issued together instead of one round trip each
#pragma unroll
    for (int it = 0; it < (RB * CPR + NT - 1) / NT; ++it) {
      const int idx = tid + it * NT;
      if (RB * CPR % NT != 0 && idx >= RB * CPR) continue;
      const int r = idx / CPR, cc = idx % CPR;
      const int m = m0 + rb * RB + r;
      if (m >= M) continue;
      const int n = n0 + cc * EPC;
      float v[EPC];
#pragma unroll
      for (int e = 0; e < EPC; e += 4) {
        const float4 a = *reinterpret_cast<const float4*>(lds + r * PITCH + (cc * EPC + e) * 4);
        v[e] = a.x; v[e + 1] = a.y; v[e + 2] = a.z; v[e + 3] = a.w;
      }
      if constexpr (Q == Quant::Int8) {
#pragma unroll
        for (int e = 0; e < EPC; ++e) v[e] *= f16_bits_to_f32(qs[n + e]);
      }
      const int rl = rb * RB + r, cl = cc * EPC;  // row and column within the tile
      if constexpr ((LN & kLnX) != 0) {
        // sum_k LN(x)_k W_nk = rstd * (sum_k x_k W'_nk - mean * u_n) + (W beta)_n, with
        // W'_nk = gamma_k W_nk; the (W beta)_n term is part of the folded bias
        const float2 st = mrg[rl];
#pragma unroll
        for (int e = 0; e < EPC; e += 4) {
          const float4 u = *reinterpret_cast<const float4*>(vec + BN + cl + e);
          v[e] = st.y * fmaf(-st.x, u.x, v[e]);
          v[e + 1] = st.y * fmaf(-st.x, u.y, v[e + 1]);
          v[e + 2] = st.y * fmaf(-st.x, u.z, v[e + 2]);
          v[e + 3] = st.y * fmaf(-st.x, u.w, v[e + 3]);
        }
      }
      if constexpr (E != Epi::None) {
#pragma unroll
        for (int e = 0; e < EPC; e += 4) {
          const float4 bb = STAGED ? *reinterpret_cast<const float4*>(vec + cl + e)
                                   : *reinterpret_cast<const float4*>(p.bias + n + e);
          v[e] += bb.x; v[e + 1] += bb.y; v[e + 2] += bb.z; v[e + 3] += bb.w;
        }
      }
      if constexpr (E == Epi::BiasGelu) {
#pragma unroll
        for (int e = 0; e < EPC; ++e) v[e] = gelu_erf(v[e]);
      }
      if constexpr (E == Epi::BiasResidual) {
        float rr[EPC];
        if (ES == 2 && p.y_f32) {  // an f32 residual beside an f32 output: from global memory
          const float4* rf = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(p.residual) +
                                                             (size_t)m * N + n);
#pragma unroll
          for (int e = 0; e < EPC; e += 4) {
            const float4 a = rf[e / 4];
            rr[e] = a.x; rr[e + 1] = a.y; rr[e + 2] = a.z; rr[e + 3] = a.w;
          }
        } else if constexpr (STAGED) {
          Vec16<T>::load(reinterpret_cast<const T*>(epi + lay.res_off + rl * (BN * 2) + cc * 16), rr);
        } else {
          Vec16<T>::load(res + (size_t)m * N + n, rr);
        }
        if constexpr ((LN & kLnRes) != 0) {
          const float2 st = mrg[BM + rl];
#pragma unroll
          for (int e = 0; e < EPC; e += 4) {
            const float4 g = *reinterpret_cast<const float4*>(vec + 2 * BN + cl + e);
            const float4 b = *reinterpret_cast<const float4*>(vec + 3 * BN + cl + e);
            rr[e] = fmaf((rr[e] - st.x) * st.y, g.x, b.x);
            rr[e + 1] = fmaf((rr[e + 1] - st.x) * st.y, g.y, b.y);
            rr[e + 2] = fmaf((rr[e + 2] - st.x) * st.y, g.z, b.z);
            rr[e + 3] = fmaf((rr[e + 3] - st.x) * st.y, g.w, b.w);
          }
        }
#pragma unroll
        for (int e = 0; e < EPC; ++e) v[e] += rr[e];
      }
      if constexpr ((LN & kLnOut) != 0) {
        // Partial statistics of the stored (rounded) values over the 64
        // columns of this chunk's 8-lane group (lanes 8j .. 8j+7 hold the
        // consecutive 16-byte chunks of one row; a group is all in or all out).
        const uint4 w = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                                   pack_bf16x2(v[6], v[7]));
        *reinterpret_cast<uint4*>(y + (size_t)m * N + n) = w;
        const uint32_t wv[4] = {w.x, w.y, w.z, w.w};
        float f[8], sum = 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          f[2 * i] = __uint_as_float(wv[i] << 16);
          f[2 * i + 1] = __uint_as_float(wv[i] & 0xffff0000u);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) sum += f[e];
        const float mean = dpp_sum8(sum) * (1.0f / 64.0f);
        float m2 = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) m2 = fmaf(f[e] - mean, f[e] - mean, m2);
        m2 = dpp_sum8(m2);
        if ((cc & 7) == 0) p.y_stats[(size_t)m * (N >> 6) + (n >> 6)] = make_float2(mean, m2);
      } else if (ES == 2 && p.y_f32) {
        float4* yf = reinterpret_cast<float4*>(reinterpret_cast<float*>(p.y) + (size_t)m * N + n);
#pragma unroll
        for (int e = 0; e < EPC; e += 4) yf[e / 4] = make_float4(v[e], v[e + 1], v[e + 2], v[e + 3]);
      } else {
        Vec16<T>::store(y + (size_t)m * N + n, v);
      }
    }
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

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// Requests the block's epilogue operands (EpiLayout) into LDS at `epi`, one
// 1 KB DMA block at a time, spread over the block's NW waves.  Rows at or past
// M read row M-1 (as the operand stages do); statistics are read as one
// contiguous run per block, clamped to the last whole 16 bytes of row M-1.
template <int BM, int BN, Epi E, int LN, int NW>
__device__ __forceinline__ void issue_epilogue_operands(const GemmParams& p, int m0, int n0, int M, uint8_t* epi,
                                                        int wave, int lane) {
  const EpiLayout lay = epi_layout_of<BM, BN, E, LN>(p.K, p.N);
  const uint32_t e0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)epi;
  for (int j = wave; j < lay.mrg_off / 1024; j += NW) {  // (the merged statistics are formed in place)
    const int o = j * 1024 + lane * 16;  // byte of the staged operands this lane fetches
    const uint8_t* src = nullptr;
    if (o < lay.res_off) {
      const int v = o / (BN * 4), c = (o % (BN * 4)) / 4;
      const float* vp = v == 0 ? (E != Epi::None ? p.bias : nullptr)
                               : v == 1 ? ((LN & kLnX) ? p.fold_u : nullptr)
                                        : v == 2 ? ((LN & kLnRes) ? p.res_gamma : nullptr)
                                                 : ((LN & kLnRes) ? p.res_beta : nullptr);
      if (vp) src = reinterpret_cast<const uint8_t*>(vp + n0 + c);
    } else if (o < lay.xst_off) {
      // (an f32 residual is read by the epilogue itself)
      const int b = o - lay.res_off, r = b / (BN * 2);
      if (!p.y_f32)
        src = reinterpret_cast<const uint8_t*>(p.residual) + ((size_t)min(m0 + r, M - 1) * p.N + n0) * 2 + b % (BN * 2);
    } else if (o < lay.mrg_off) {
      const bool xs = o < lay.rst_off;
      const int np = xs ? p.K >> 6 : p.N >> 6;
      const size_t b = (size_t)m0 * np * 8 + (o - (xs ? lay.xst_off : lay.rst_off));
      src = reinterpret_cast<const uint8_t*>(xs ? p.x_stats : p.res_stats) + min(b, (size_t)M * np * 8 - 16);
    }
    if (src) lds_dma16(src, __builtin_amdgcn_readfirstlane(e0 + j * 1024));
  }
}

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
  return q == Quant::None || q == Quant::Int8 || q == Quant::Int8G || q == Quant::Int4 || q == Quant::Int4M;
}
__host__ __device__ constexpr bool quant_grouped(Quant q) {
  return q == Quant::Int8G || q == Quant::Int4 || q == Quant::Int4M;
}
// LDS for the group scales (and zeros / mins) of BN rows over K.
__host__ __device__ inline int gq_lds_bytes(Quant q, int BN, int K) {
  return quant_grouped(q) ? (BN * (K / 32) * 2 * (q == Quant::Int8G ? 1 : 2) + 1023) / 1024 * 1024 : 0;
}

template <int BM, int BN, int STAGES, typename T, Epi E, int KS = 1, int LN = 0, Quant Q = Quant::None>
__global__ __launch_bounds__(kThreads * KS) void gemm_dma_kernel(GemmParams p) {
  static_assert(BM % 64 == 0 && BN % 64 == 0 && STAGES >= 2 && STAGES <= 6, "tile");
  static_assert(KS == 1 || (sizeof(T) == 2 && (BK_BF16 / 16) % KS == 0), "K split over bf16 chunks");
  static_assert(dma_quant_ok(Q) && (Q == Quant::None || (sizeof(T) == 2 && LN == 0)), "quantised: bf16, no LN");
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
  // oldest in every wave's memory queue: landed before the first stage is waited for
  if constexpr (STAGED) issue_epilogue_operands<BM, BN, E, LN, NW>(p, m0, n0, M, epi_lds, wave, lane);
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

  // Group scales (then zeros / mins) of rows n0 .. n0+BN-1, [BN][K/32] f16
  // each, into LDS after the epilogue operands: older than every stage load,
  // so the first stage's wait covers them.
  const int G = K / 32;
  uint8_t* gq = epi_lds + (STAGED ? epi_layout_of<BM, BN, E, LN>(p.K, p.N).bytes : 0);
  if constexpr (quant_grouped(Q)) {
    const int dw = BN * G / 2;  // dwords per array (G is even)
    const uint32_t gq0 = lds_addr_of(gq);
    for (int a = 0; a < (Q == Quant::Int8G ? 1 : 2); ++a) {
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

#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < KT) issue(st, st);

  for (int kt0 = 0; kt0 < KT; kt0 += STAGES) {
#pragma unroll
    for (int u = 0; u < STAGES; ++u) {
      const int kt = kt0 + u;
      if (kt < KT) {
        if (NI % NW == 0 || wave < NI % NW)
          wait_stage<LPS, STAGES - 2>(min(STAGES - 2, KT - 1 - kt));
        else
          wait_stage<(NI % NW == 0 ? LPS : LPS - 1), STAGES - 2>(min(STAGES - 2, KT - 1 - kt));
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
  store_tile<BM, BN, T, Q, E, TM, TN, NRB, KS, LN, STAGED>(acc, smem, p, m0, n0, M, epi_lds);
}

template <int BM, int BN, int STAGES, typename T, Epi E, int KS, int LN, Quant Q = Quant::None>
hipError_t launch_dma(const GemmParams& p, hipStream_t s) {
  const dim3 grid((p.N / BN) * ((p.M + BM - 1) / BM));
  const size_t epi = (sizeof(T) == 2 ? (size_t)epi_layout_of<BM, BN, E, LN>(p.K, p.N).bytes : 0) +
                     (size_t)gq_lds_bytes(Q, BN, p.K);
  hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, STAGES, T, E, KS, LN, Q>), grid, dim3(kThreads * KS), epi, s, p);
  return hipGetLastError();
}

// Quantised weights through the DMA kernel (bf16 activations, no deferred
// LayerNorm): 64 x 128 tiles for the wide projections, else 64 x 64.
template <int BM, int BN, int STAGES, Quant Q>
hipError_t launch_dma_q_tile(const GemmParams& p, hipStream_t s) {
  switch (p.epi) {
    case Epi::None: return launch_dma<BM, BN, STAGES, bf16_t, Epi::None, 1, 0, Q>(p, s);
    case Epi::Bias: return launch_dma<BM, BN, STAGES, bf16_t, Epi::Bias, 1, 0, Q>(p, s);
    case Epi::BiasGelu: return launch_dma<BM, BN, STAGES, bf16_t, Epi::BiasGelu, 1, 0, Q>(p, s);
    case Epi::BiasResidual: return launch_dma<BM, BN, STAGES, bf16_t, Epi::BiasResidual, 1, 0, Q>(p, s);
  }
  return hipErrorInvalidValue;
}

// The group scales of a tile's rows must fit the LDS next to the ring: up to
// 32 KB (for example K <= 4096 with 64 weight rows of int4 scales and zeros),
// and come by dword DMA, so 4-byte aligned; otherwise the register-staged
// kernel runs.
bool dma_q_fits(const GemmParams& p, int BN) {
  auto a4 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 3) == 0; };
  if (quant_grouped(p.quant) && (!a4(p.scales) || (p.quant != Quant::Int8G && !a4(p.zeros)))) return false;
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
template <Quant Q>
hipError_t launch_dma_q(const GemmParams& p, hipStream_t s) {
  if (p.K >= 1024) {
    if (p.N % 128 == 0 && p.N >= 1024 && dma_q_fits(p, 128)) return launch_dma_q_tile<64, 128, 4, Q>(p, s);
    if (dma_q_fits(p, 64)) return launch_dma_q_tile<64, 64, 5, Q>(p, s);
  }
  return launch_typed<bf16_t, Q>(p, s);
}

template <int BM, int BN, int STAGES, typename T, int KS = 1>
hipError_t launch_dma_tile(const GemmParams& p, hipStream_t s) {
  const int ln = (p.x_stats ? kLnX : 0) | (p.res_stats ? kLnRes : 0) | (p.y_stats ? kLnOut : 0);
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

}  // namespace

hipError_t launch_fold_ln_weights(const void* w, int N, int K, const float* gamma, const float* beta,
                                  const float* bias, void* w_out, float* u_out, float* v_out, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  hipLaunchKernelGGL(fold_ln_weights_kernel, dim3(N), dim3(256), 0, s, reinterpret_cast<const bf16_t*>(w), K, gamma,
                     beta, bias, reinterpret_cast<bf16_t*>(w_out), u_out, v_out);
  return hipGetLastError();
}

bool gemm_deferred_ln_supported(DType dt, Quant q, int H) {
  // rows of an even number of 64-column parts (whole 16-byte statistics runs), up to 1024 columns
  return dt == DType::BF16 && q == Quant::None && H % 128 == 0 && H <= 64 * kLnMaxParts;
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
    case Quant::Int4M: return launch_dma_q<Quant::Int4M>(p, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_dequant_unpack(const void* w, Quant q, const void* scales, const void* zeros, int N, int K,
                                 float* out, hipStream_t s) {
  const size_t total = (size_t)N * K;
  const int blocks = (int)std::min<size_t>((total + 255) / 256, 4096);
  hipLaunchKernelGGL(dequant_unpack_kernel, dim3(blocks), dim3(256), 0, s, reinterpret_cast<const uint8_t*>(w), q,
                     reinterpret_cast<const uint16_t*>(scales), reinterpret_cast<const uint16_t*>(zeros), N, K, out);
  return hipGetLastError();
}

}  // namespace rlx
