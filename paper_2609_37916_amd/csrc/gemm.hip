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
//    Stages are double-buffered in LDS with 16 bytes of padding per row so
//    that the 16-byte fragment reads of 16 consecutive rows hit distinct banks.
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
#include "common.hpp"
#include "kernels.hpp"

namespace rlx {
namespace {

constexpr int kThreads = 256;
constexpr int kRowBytes = 128;            // bytes of one operand row per K stage
constexpr int kLdsRow = kRowBytes + 16;   // padded LDS row pitch in bytes

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
  constexpr int WCPR = Q == Quant::None ? 8 : (Q == Quant::Int8 ? 4 : 2);
  constexpr int WLDS = Q == Quant::None ? 16 : (Q == Quant::Int8 ? 32 : 64);
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
  const size_t w_pitch = Q == Quant::None ? (size_t)K * ES : (Q == Quant::Int8 ? (size_t)K : (size_t)K / 2);
  const int wk_bytes = Q == Quant::None ? kRowBytes : (Q == Quant::Int8 ? 64 : 32);  // weight bytes per row per stage

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

  // Epilogue: lane owns row m = l32 of each m-tile and columns
  // n = 8*i + 4*half + j (j = 0..3) of each n-tile, register 4*i + j.
  const int N = p.N;
  T* y = reinterpret_cast<T*>(p.y);
  const T* res = reinterpret_cast<const T*>(p.residual);
  const uint16_t* qs = reinterpret_cast<const uint16_t*>(p.scales);
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int m = m0 + wm * WM + tm * 32 + l32;
    if (m >= M) continue;
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int n = n0 + wn * WN + tn * 32 + i * 8 + half * 4;
        float v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = acc[tm][tn][4 * i + j];
        if constexpr (Q == Quant::Int8) {
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] *= f16_bits_to_f32(qs[n + j]);
        }
        if constexpr (E != Epi::None) {
          float4 bb = *reinterpret_cast<const float4*>(p.bias + n);
          v[0] += bb.x; v[1] += bb.y; v[2] += bb.z; v[3] += bb.w;
        }
        if constexpr (E == Epi::BiasGelu) {
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = gelu_erf(v[j]);
        }
        if constexpr (E == Epi::BiasResidual) {
          float r[4];
          OutVec<T>::load4(res + (size_t)m * N + n, r);
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] += r[j];
        }
        OutVec<T>::store4(y + (size_t)m * N + n, v);
      }
    }
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
    } else {
      const uint8_t byte = w[(size_t)n * (K / 2) + k / 2];
      const float code = (float)((k & 1) ? (byte >> 4) : (byte & 0xf));
      const size_t g = (size_t)n * (K / 32) + k / 32;
      out[i] = (code - f16_bits_to_f32(zeros[g])) * f16_bits_to_f32(scales[g]);
    }
  }
}

}  // namespace

hipError_t launch_gemm(const GemmParams& p, hipStream_t s) {
  if (p.M <= 0) return hipSuccess;
  if (p.dtype == DType::F32) return launch_typed<float, Quant::None>(p, s);
  switch (p.quant) {
    case Quant::None: return launch_typed<bf16_t, Quant::None>(p, s);
    case Quant::Int8: return launch_typed<bf16_t, Quant::Int8>(p, s);
    case Quant::Int4: return launch_typed<bf16_t, Quant::Int4>(p, s);
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
