// QKV projection fused with masked attention for one (sequence, head) of at
// most 128 tokens, bf16, dense weights, head_dim 32 -- the block body shared by
// the standalone kernel (attention.hip) and the persistent encoder forward
// (pipe.hip).  The paper fuses the attention block and reads Q, K and V as
// strided narrows of one projection (Section III-B); here the narrow of one
// head is computed in the block itself and never leaves the chip.
//
// Phase 1 computes the sequence's 96 projection columns of this head (32 each
// of Q, K, V; K = H) with the LDS-DMA pipeline of the dense GEMM; wave w owns
// tokens 32w .. 32w+31.  Phase 2 is the attention over those rows.  Q stays in
// registers -- its MFMA output layout (token = lane % 32, head dims
// 8i + 4*(lane/32) + j) is directly a valid operand order, as long as K is read
// back in the same dim order -- while K (row-major) and V (transposed) go
// through LDS for the other waves.  The context is written head-major
// ([head][token][32]), so each wave's output is one contiguous 2 KB block; the
// output projection reads that layout.
#pragma once
#include "common.hpp"
#include "kernels.hpp"

namespace rlx {
namespace {

constexpr int kFxRows = 128;               // token rows of the stage (max sequence length)
constexpr int kFwRows = 96;                // projection columns of one head
constexpr int kFRow = 128;                 // bytes per staged row (64 k of bf16)
constexpr int kFStage = (kFxRows + kFwRows) * kFRow;
constexpr int kFLps = (kFxRows + kFwRows) / 32;   // DMA instructions per thread per stage (7)
constexpr int kFXLps = kFxRows / 32;       // of which token rows (4); the rest are weight rows
constexpr int kFKPitch = 72;               // bytes per K row in LDS (64 + 8): conflict-free 8-byte reads
constexpr int kFVts = 132;                 // V^T row pitch in elements (264 bytes)
constexpr int kFOutOff = 20480;            // per-wave 2 KB output staging, after K and V^T
constexpr float kFLog2e = 1.4426950408889634f;

// LDS of one block: the stage ring (1 KB aligned), this head's bias then
// fold_u values [2][96] f32, and the sequence's partial row statistics
// [128][kLnMaxParts] float2.
template <int STAGES>
constexpr int qkv_attention_ring_bytes() { return STAGES * kFStage; }
constexpr int kFVecBytes = 2 * kFwRows * 4;
constexpr int kFStatBytes = kFxRows * kLnMaxParts * 8;

__device__ __forceinline__ int fswz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// The sequence occupies rows row0 .. row0+L-1 of p.x (1 <= L <= 128).
// wait_inputs() is called by every thread after the head's weight rows of
// the first stages (and its bias / fold_u values) have been requested and
// before anything that depends on the rows of x or their statistics is
// requested; when it returns, those inputs must be visible to every thread
// (a no-op when they were written by an earlier kernel).  All threads return.
template <int STAGES, typename Wait>
__device__ __forceinline__ void qkv_attention_block(const FusedAttnParams& p, int row0, int L, int h, uint8_t* smem,
                                                    float* vec_lds, float2* st_lds, Wait&& wait_inputs) {
  static_assert(STAGES >= 2 && STAGES <= 4, "stages");
  static_assert(kFxRows * kFKPitch + 32 * kFVts * 2 <= kFOutOff, "K/V before the output staging");
  static_assert(STAGES * kFStage >= kFOutOff + 4 * 2048, "K/V and output staging reuse the stage memory");
  // block-uniform values, made scalar so every loop holding a barrier has a
  // scalar trip count
  const int H = __builtin_amdgcn_readfirstlane(p.H);
  row0 = __builtin_amdgcn_readfirstlane(row0);
  L = __builtin_amdgcn_readfirstlane(L);
  h = __builtin_amdgcn_readfirstlane(h);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const bool active = wave * 32 < L;
  const size_t pitch = (size_t)H * 2;
  const bool deferred = p.x_stats != nullptr;
  const int np = H >> 6;
  const int KT = H / 64;

  // DMA sources: instruction i of a wave fills stage rows wave*8 + 32i .. +7;
  // rows < 128 are token rows (clamped to the sequence), the rest this head's
  // 96 weight rows (Q, K, V parts).
  const uint8_t* src[kFLps];
#pragma unroll
  for (int i = 0; i < kFLps; ++i) {
    const int row = wave * 8 + i * 32 + (lane >> 3);
    const int c = fswz(row, lane & 7);
    const uint8_t* base;
    if (row < kFxRows) {
      base = reinterpret_cast<const uint8_t*>(p.x) + (size_t)(row0 + min(row, L - 1)) * pitch;
    } else {
      const int n = row - kFxRows;
      base = reinterpret_cast<const uint8_t*>(p.wqkv) + (size_t)((n >> 5) * H + h * 32 + (n & 31)) * pitch;
    }
    src[i] = base + c * 16;
  }
  const uint32_t lds0 = lds_addr_of(smem);
  auto issue_part = [&](int kt, int buf, int i0, int i1) {
#pragma unroll
    for (int i = 0; i < kFLps; ++i) {
      if (i < i0 || i >= i1) continue;
      const uint32_t la = lds0 + buf * kFStage + (wave * 8 + i * 32) * kFRow;
      lds_dma16(src[i] + (size_t)kt * kFRow, __builtin_amdgcn_readfirstlane(la));
    }
  };

  // 1. Weights, which depend on nothing: this head's 96 bias values and
  //    (deferred LayerNorm input) 96 row sums of the gamma-scaled weights,
  //    eight lanes per 32-value segment, then the weight rows of the first
  //    stages.
  if (wave == 0 && lane < (deferred ? 48 : 24)) {
    const int seg = lane >> 3, part = seg % 3;  // segments 0-2: bias Q, K, V; 3-5: fold_u Q, K, V
    const float* vp = (seg < 3 ? p.bqkv : p.fold_u) + part * H + h * 32 + (lane & 7) * 4;
    lds_dma16(vp, __builtin_amdgcn_readfirstlane(lds_addr_of(vec_lds)));
  }
#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < KT) issue_part(st, st, kFXLps, kFLps);
  wait_inputs();
  // 2. The sequence's row statistics (one contiguous run clamped to its last
  //    row) and token rows.
  if (deferred) {
    const uint32_t s0 = lds_addr_of(st_lds);
    const size_t first = (size_t)row0 * np * 8, end = (size_t)(row0 + L) * np * 8;
    const int jobs = (L * np * 8 + 1023) >> 10;
    for (int j = wave; j < jobs; j += 4) {
      const size_t o = min(first + (size_t)j * 1024 + lane * 16, end - 16);
      lds_dma16(reinterpret_cast<const uint8_t*>(p.x_stats) + o, __builtin_amdgcn_readfirstlane(s0 + j * 1024));
    }
  }
#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < KT) issue_part(st, st, 0, kFXLps);

  // (0, 1) leaves a plain input's product as is
  float2 lnst = make_float2(0.0f, 1.0f);
  f32x16_t acc[3];
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[t][v] = 0.0f;

  for (int kt0 = 0; kt0 < KT; kt0 += STAGES) {
#pragma unroll
    for (int u = 0; u < STAGES; ++u) {
      const int kt = kt0 + u;
      if (kt < KT) {
        // stage 0: everything requested so far (its weight rows went out first)
        const int ahead = kt == 0 ? 0 : min(STAGES - 2, KT - 1 - kt);
        if (STAGES >= 4 && ahead >= 2) wait_vmcnt<2 * kFLps>();
        else if (STAGES >= 3 && ahead >= 1) wait_vmcnt<kFLps>();
        else wait_vmcnt<0>();
        __syncthreads();
        if (kt + STAGES - 1 < KT) issue_part(kt + STAGES - 1, (u + STAGES - 1) % STAGES, 0, kFLps);
        if (active) {
          const uint8_t* xs = smem + u * kFStage;
          const uint8_t* ws = xs + kFxRows * kFRow;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int rx = wave * 32 + l32;
            const bf16x8_t xf = as_bf16x8(*reinterpret_cast<const uint4*>(xs + rx * kFRow + fswz(rx, 2 * q + half) * 16));
#pragma unroll
            for (int t = 0; t < 3; ++t) {
              const int rw = t * 32 + l32;
              const bf16x8_t wf =
                  as_bf16x8(*reinterpret_cast<const uint4*>(ws + rw * kFRow + fswz(rw, 2 * q + half) * 16));
              acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf, xf, acc[t], 0, 0, 0);
            }
          }
          // (mean, rstd) of this lane's token, while the first stage's MFMAs
          // run: the statistics were requested before stage 0 and the stage-0
          // barrier published them
          if (kt == 0 && deferred) lnst = merge_ln_lds(st_lds + min(wave * 32 + l32, L - 1) * np, np, p.ln_eps);
        }
      }
    }
  }
  __syncthreads();  // all waves are done with the stage buffers: K and V^T reuse them

  uint8_t* k_lds = smem;                                               // [128][72 B]
  bf16_t* vt_lds = reinterpret_cast<bf16_t*>(smem + kFxRows * kFKPitch);  // [32][kFVts]
  // Register v of acc[t] holds token 32*wave + l32, head dim 8*(v/4) + 4*half + (v%4) of part t.
  uint32_t qpk[8];
  if (active) {
    const int tok = wave * 32 + l32;
    // this lane's bias and (deferred input) fold_u values, every LDS read
    // issued at once: vector reads of 4 dims per part; fold_u is zero for a
    // plain input, so the loop below has no branch
    float4 bb[3][4], uu[3][4];
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        bb[t][i] = *reinterpret_cast<const float4*>(vec_lds + 32 * t + 8 * i + 4 * half);
        uu[t][i] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    if (deferred) {
#pragma unroll
      for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) uu[t][i] = *reinterpret_cast<const float4*>(vec_lds + kFwRows + 32 * t + 8 * i + 4 * half);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d = 8 * i + 4 * half;
      float out[3][4];
      // deferred LayerNorm of the input rows: sum_k LN(x)_k W_nk =
      // rstd * (sum_k x_k W'_nk - mean * u_n) + (W beta)_n, W'_nk = gamma_k W_nk
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const float b4[4] = {bb[t][i].x, bb[t][i].y, bb[t][i].z, bb[t][i].w};
        const float u4[4] = {uu[t][i].x, uu[t][i].y, uu[t][i].z, uu[t][i].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) out[t][j] = fmaf(lnst.y, fmaf(-lnst.x, u4[j], acc[t][4 * i + j]), b4[j]);
      }
      qpk[2 * i] = pack_bf16x2(out[0][0], out[0][1]);
      qpk[2 * i + 1] = pack_bf16x2(out[0][2], out[0][3]);
      *reinterpret_cast<uint2*>(k_lds + tok * kFKPitch + d * 2) =
          make_uint2(pack_bf16x2(out[1][0], out[1][1]), pack_bf16x2(out[1][2], out[1][3]));
#pragma unroll
      for (int j = 0; j < 4; ++j) vt_lds[(d + j) * kFVts + tok] = f32_to_bf16(out[2][j]);
    }
  }
  __syncthreads();
  if (active) {
    const int ntiles = (L + 31) >> 5;
    const bf16x8_t qf0 = as_bf16x8(make_uint4(qpk[0], qpk[1], qpk[2], qpk[3]));
    const bf16x8_t qf1 = as_bf16x8(make_uint4(qpk[4], qpk[5], qpk[6], qpk[7]));
    const float sl2 = p.scale * kFLog2e;
    float l_run = 0.0f;
    f32x16_t o;
#pragma unroll
    for (int v = 0; v < 16; ++v) o[v] = 0.0f;
    // Two passes over the (at most four) key tiles, the scores kept in
    // registers: all S^T tiles first, then the row maximum over every key, then
    // P = 2^(s - max) and P.V -- no running-max rescale of the output.
    f32x16_t sc[kFxRows / 32];
#pragma unroll
    for (int t = 0; t < kFxRows / 32; ++t) {
      if (t >= ntiles) break;
      const int kb = t * 32;
      // K operand in the same head-dim order as Q: dims 4*half + {0..3} and 8 + 4*half + {0..3} (+16 for step 2)
      const uint8_t* krow = k_lds + (kb + l32) * kFKPitch + 8 * half;
      const uint2 k00 = *reinterpret_cast<const uint2*>(krow);
      const uint2 k01 = *reinterpret_cast<const uint2*>(krow + 16);
      const uint2 k10 = *reinterpret_cast<const uint2*>(krow + 32);
      const uint2 k11 = *reinterpret_cast<const uint2*>(krow + 48);
#pragma unroll
      for (int v = 0; v < 16; ++v) sc[t][v] = 0.0f;
      sc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(make_uint4(k00.x, k00.y, k01.x, k01.y)), qf0, sc[t], 0,
                                                      0, 0);
      sc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(make_uint4(k10.x, k10.y, k11.x, k11.y)), qf1, sc[t], 0,
                                                      0, 0);
    }
    // The maximum is taken over the raw scores and scaled once (the scale
    // 1/sqrt(d) is positive, so scaling keeps the order): each probability is
    // then one fma and one exp2.  Only the last key tile can be partial, so
    // only it is masked.
    float m_raw = -INFINITY;
#pragma unroll
    for (int t = 0; t < kFxRows / 32; ++t) {
      if (t >= ntiles) break;
      const int kb = t * 32;
      if (kb + 32 > L) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kb + 8 * (v >> 2) + 4 * half + (v & 3);
          if (key >= L) sc[t][v] = -INFINITY;
        }
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) m_raw = fmaxf(m_raw, sc[t][v]);
    }
    m_raw = fmaxf(m_raw, __shfl_xor(m_raw, 32, 64));  // finite: the sequence has a real key
    const float m_neg = -(m_raw * sl2);
#pragma unroll
    for (int t = 0; t < kFxRows / 32; ++t) {
      if (t >= ntiles) break;
      const int kb = t * 32;
      // v_exp_f32 directly: the arguments are <= 0 and results below 2^-126
      // (flushed to 0) are far under the bf16 rounding of P
      float pv[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) pv[v] = __builtin_amdgcn_exp2f(fmaf(sc[t][v], sl2, m_neg));
      float ps[8];
#pragma unroll
      for (int v = 0; v < 8; ++v) ps[v] = pv[2 * v] + pv[2 * v + 1];
      l_run += ((ps[0] + ps[1]) + (ps[2] + ps[3])) + ((ps[4] + ps[5]) + (ps[6] + ps[7]));
      const uint4 pb0 = make_uint4(pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]), pack_bf16x2(pv[4], pv[5]),
                                   pack_bf16x2(pv[6], pv[7]));
      const uint4 pb1 = make_uint4(pack_bf16x2(pv[8], pv[9]), pack_bf16x2(pv[10], pv[11]),
                                   pack_bf16x2(pv[12], pv[13]), pack_bf16x2(pv[14], pv[15]));
      const bf16_t* vrow = vt_lds + l32 * kFVts + kb + 4 * half;
      const uint2 v00 = *reinterpret_cast<const uint2*>(vrow);
      const uint2 v01 = *reinterpret_cast<const uint2*>(vrow + 8);
      const uint2 v10 = *reinterpret_cast<const uint2*>(vrow + 16);
      const uint2 v11 = *reinterpret_cast<const uint2*>(vrow + 24);
      o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(make_uint4(v00.x, v00.y, v01.x, v01.y)), as_bf16x8(pb0), o,
                                                  0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(make_uint4(v10.x, v10.y, v11.x, v11.y)), as_bf16x8(pb1), o,
                                                  0, 0, 0);
    }
    const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
    const float inv = 1.0f / l_tot;
    // Output block of this wave: 32 tokens x 32 dims (64-byte rows), contiguous in
    // the head-major layout.  Transpose it through LDS so the global write is
    // whole 16-byte lanes over 1 KB runs; rows past the sequence are not written
    // (they belong to the next sequence).
    uint8_t* ob = smem + kFOutOff + wave * 2048;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d = 8 * i + 4 * half;
      *reinterpret_cast<uint2*>(ob + l32 * 64 + d * 2) = make_uint2(pack_bf16x2(o[4 * i] * inv, o[4 * i + 1] * inv),
                                                                    pack_bf16x2(o[4 * i + 2] * inv, o[4 * i + 3] * inv));
    }
    __builtin_amdgcn_wave_barrier();
    uint8_t* og = reinterpret_cast<uint8_t*>(p.out) + ((size_t)h * p.out_rows + row0 + wave * 32) * 64;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int chunk = lane + 64 * j;  // 16-byte chunk of the 2 KB block; row = chunk / 4
      if (wave * 32 + (chunk >> 2) < L)
        *reinterpret_cast<uint4*>(og + chunk * 16) = *reinterpret_cast<const uint4*>(ob + chunk * 16);
    }
  }
}

}  // namespace
}  // namespace rlx
