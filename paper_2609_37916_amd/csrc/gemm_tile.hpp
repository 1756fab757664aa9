// Tile machinery shared by the GEMM kernels (gemm.hip) and the persistent
// encoder forward (pipe.hip): operand-row constants, the LDS-staged fused
// epilogue (bias, erf-GELU, residual, deferred-LayerNorm statistics, int8
// scales) and the direct-to-LDS request of a tile's epilogue operands.
#pragma once
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
// Deferred-LayerNorm roles of a bf16-activation GEMM (the GemmParams fields):
// normalise the product of a deferred input, normalise a deferred residual,
// write the partial statistics of the output.  With quantised weights, where
// gamma cannot be folded into the codes, the LayerNorm input travels
// gamma-scaled: kLnOutG stores gamma[n] * y (statistics still of y) and
// kLnResG takes a residual stored that way.
constexpr int kLnX = 1, kLnRes = 2, kLnOut = 4, kLnOutG = 8, kLnResG = 16;

// Epilogue operands staged in LDS (bf16-activation kernels): the block's per-column
// vectors [bias, fold_u, res_gamma, res_beta(, y_gamma)][BN] (f32), its residual tile
// [BM][BN] (bf16) and the partial statistics of its rows ([BM][K/64] for x,
// [BM][N/64] for the residual).  Every region is a whole number of 1 KB DMA
// blocks.  They are requested before the first operand stage, so by the
// epilogue they have long landed and the epilogue reads no global memory.
// The statistics regions are followed by the rows' merged (mean, rstd)
// ([2][BM] float2: x, residual), which the epilogue forms once per row: a
// row's merge reads kLnMaxParts entries (128 bytes) at once, so the last row's
// read may run up to 128 bytes past its region, into the next region or the
// merged statistics -- always inside the allocation, and masked.
struct EpiLayout {
  int res_off, xst_off, rst_off, mrg_off, bytes;
};
__host__ __device__ constexpr EpiLayout epi_layout(int BM, int BN, bool res, bool xst, bool rst, int K, int N,
                                                   bool out_gamma = false) {
  EpiLayout L{};
  int off = out_gamma ? (20 * BN + 1023) / 1024 * 1024 : 16 * BN;  // four (five) f32 vectors of BN
  L.res_off = off;
  if (res) off += BM * BN * 2;
  L.xst_off = off;
  if (xst) off += (BM * (K / 64) * 8 + 1023) / 1024 * 1024;
  L.rst_off = off;
  if (rst) off += (BM * (N / 64) * 8 + 1023) / 1024 * 1024;
  L.mrg_off = off;
  if (xst || rst) off += (2 * BM * 8 + 1023) / 1024 * 1024;
  L.bytes = off;
  return L;
}
template <int BM, int BN, Epi E, int LN>
__host__ __device__ constexpr EpiLayout epi_layout_of(int K, int N) {
  return epi_layout(BM, BN, E == Epi::BiasResidual, (LN & kLnX) != 0, (LN & kLnRes) != 0, K, N,
                    (LN & kLnOutG) != 0);
}

// Merges the partial statistics staged at `epi` into each row's (mean, rstd)
// at the EpiLayout's mrg region: x rows at [0, BM), residual rows at [BM, 2BM).
// One thread per row: thread `tid` of 0 .. BM-1 merges row tid, others none.
template <int BM, int BN, Epi E, int LN>
__device__ __forceinline__ void merge_row_stats(const GemmParams& p, uint8_t* epi, int tid) {
  if constexpr ((LN & (kLnX | kLnRes)) != 0) {
    const EpiLayout lay = epi_layout_of<BM, BN, E, LN>(p.K, p.N);
    float2* mrg = reinterpret_cast<float2*>(epi + lay.mrg_off);
    if (tid >= 0 && tid < BM) {
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
  static_assert(LN == 0 || (sizeof(T) == 2 && STAGED), "deferred LayerNorm: bf16 activations, staged operands");
  static_assert(!(LN & kLnOutG) || (LN & kLnOut), "gamma-scaled output: with its statistics");
  static_assert(!(LN & kLnResG) || (LN & kLnRes), "gamma-scaled residual: a deferred residual");
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
  const float* vec = reinterpret_cast<const float*>(epi);  // [4 or 5][BN]: bias, fold_u, res_gamma, res_beta, y_gamma
  float2* mrg = reinterpret_cast<float2*>(epi + lay.mrg_off);  // [2][BM]: (mean, rstd) of x rows, residual rows
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    __syncthreads();  // the operand stages (or the previous row block) are no longer read
    // the block's last BM threads merge the rows' statistics (one row each)
    // while the other waves stage their accumulators; the barrier after the
    // staging publishes them
    if (rb == 0) merge_row_stats<BM, BN, E, LN>(p, epi, tid - (NT - BM));
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
            if constexpr ((LN & kLnResG) != 0) {  // stored gamma * a: rstd * (r - mean * gamma) + beta
              rr[e] = fmaf(fmaf(-st.x, g.x, rr[e]), st.y, b.x);
              rr[e + 1] = fmaf(fmaf(-st.x, g.y, rr[e + 1]), st.y, b.y);
              rr[e + 2] = fmaf(fmaf(-st.x, g.z, rr[e + 2]), st.y, b.z);
              rr[e + 3] = fmaf(fmaf(-st.x, g.w, rr[e + 3]), st.y, b.w);
            } else {
              rr[e] = fmaf((rr[e] - st.x) * st.y, g.x, b.x);
              rr[e + 1] = fmaf((rr[e + 1] - st.x) * st.y, g.y, b.y);
              rr[e + 2] = fmaf((rr[e + 2] - st.x) * st.y, g.z, b.z);
              rr[e + 3] = fmaf((rr[e + 3] - st.x) * st.y, g.w, b.w);
            }
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
        if constexpr ((LN & kLnOutG) != 0) {  // stored: gamma * y, each rounded once
          const float4 g0 = *reinterpret_cast<const float4*>(vec + 4 * BN + cl);
          const float4 g1 = *reinterpret_cast<const float4*>(vec + 4 * BN + cl + 4);
          *reinterpret_cast<uint4*>(y + (size_t)m * N + n) =
              make_uint4(pack_bf16x2(g0.x * v[0], g0.y * v[1]), pack_bf16x2(g0.z * v[2], g0.w * v[3]),
                         pack_bf16x2(g1.x * v[4], g1.y * v[5]), pack_bf16x2(g1.z * v[6], g1.w * v[7]));
        } else {
          *reinterpret_cast<uint4*>(y + (size_t)m * N + n) = w;
        }
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
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// Requests the block's epilogue operands (EpiLayout) into LDS at `epi`, one
// 1 KB DMA block at a time, spread over the block's NW waves.  Rows at or past
// M read row M-1 (as the operand stages do); statistics are read as one
// contiguous run per block, clamped to the last whole 16 bytes of row M-1.
// With EXACT, every block is one DMA instruction of the wave, also where some
// or all of its lanes have no operand (they fetch 16 bytes of the weights
// into a slot nothing reads), so the wave's count of loads is exactly
// epilogue_dma_count(): callers may wait for older loads with it.
template <int BM, int BN, Epi E, int LN, int NW>
__device__ __forceinline__ int epilogue_dma_count(const GemmParams& p, int wave) {
  const int nb = epi_layout_of<BM, BN, E, LN>(p.K, p.N).mrg_off / 1024;
  return wave < nb ? (nb - wave + NW - 1) / NW : 0;
}
template <int BM, int BN, Epi E, int LN, int NW, bool EXACT = false>
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
                               : v == 3 ? ((LN & kLnRes) ? p.res_beta : nullptr)
                               : v == 4 ? ((LN & kLnOutG) ? p.y_gamma : nullptr)
                                        : nullptr;  // (the padding of the vector region)
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
    if constexpr (EXACT)
      lds_dma16(src ? src : reinterpret_cast<const uint8_t*>(p.w), __builtin_amdgcn_readfirstlane(e0 + j * 1024));
    else if (src)
      lds_dma16(src, __builtin_amdgcn_readfirstlane(e0 + j * 1024));
  }
}


}  // namespace
}  // namespace rlx
