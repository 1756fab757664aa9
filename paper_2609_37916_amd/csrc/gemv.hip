// Dequantising matmul for a few activation rows (the GEMV regime of
// Op::DequantMatMul, Section VI; Linear block, Section III-A):
//
//   y[m, n] = epi( sum_k x[m, k] W[n, k] ),   1 <= M <= 16 bf16 rows,
//
// with W in the int8 per-channel or the int4 group-32 zero-point layout.
// With so few rows the product reads every weight byte once and does little
// arithmetic per byte: it is bound by HBM bandwidth and by the vector-ALU
// work of unpacking the codes, not by the matrix cores.
//
//  * One block per 16 output columns.  Its 8 waves split K in 128-k units
//    (unit u goes to wave u mod 8); the 8 partial 16 x 16 tiles are added in
//    LDS in wave order (deterministic) before the epilogue.
//  * Each wave streams its units through a private ring of LDS slots with
//    direct-to-LDS loads, four units in flight, so the K loop needs no
//    barrier.  A unit's 16 weight rows land group-major ([16-byte chunk]
//    [row][16 B]): lane (n, G) then reads the 4 (int4) or 8 (int8) bytes of
//    k-octet G of each group with conflict-free ds_read2.
//  * v_mfma_f32_16x16x32_bf16 takes the activations as the A operand (rows m;
//    rows M..15 repeat row M-1 and their results are dropped) and the codes
//    as B, one 32-k group per instruction.  Lane l supplies row / column
//    l % 16 and k-octet G = l / 16 of the group; its eight bf16 slots pair
//    k = 8G + i with 8G + i + 4 (i = 0..3), the pairing the nibble unpacking
//    yields at the lowest cost.  The activations are stored in LDS in that
//    order once per block, with the per-group sums X[m, g] = sum_k x[m, k].
//  * int4: nibble q becomes the bf16 value 128 + q with one AND-OR (0x4300,
//    the exponent of 128, over the nibble), so a group's instruction gives
//    V = sum_k x_k (128 + q_k) and the group contributes
//    s V - s (128 + z) X.  The s V terms are added per group with four FMAs
//    a lane; the s (128 + z) X terms of four groups are one
//    v_mfma_f32_16x16x4_f32 (X as A, -s (128 + z) as B).  No weight is
//    rounded: every rounding is an fp32 sum (the tiled path instead rounds
//    each (q - z) s to bf16).
//  * int8: codes convert exactly to bf16 and one accumulator takes every
//    group; the per-channel scale multiplies the fp32 sum in the epilogue, as
//    in the tiled path.
#include "common.hpp"
#include "kernels.hpp"

namespace rlx {
namespace {

constexpr int kGvWaves = 8;
constexpr int kGvThreads = kGvWaves * 64;
constexpr int kGvUnitK = 128;       // k per unit (four 32-k groups)
constexpr int kGvDepth = 4;         // units in flight per wave
constexpr int kGvMaxRows = 16;
constexpr int kGvMaxXBytes = 64 * 1024;  // activations staged in LDS (bf16)

template <Quant Q>
struct GvUnit;
template <>
struct GvUnit<Quant::Int4> {
  // codes: 16 rows x 64 bytes; meta: scales then zeros, 16 rows x 4 f16 each
  static constexpr int kCodeBytes = 1024, kMetaBytes = 256, kLoads = 2;
};
template <>
struct GvUnit<Quant::Int8> {
  static constexpr int kCodeBytes = 2048, kMetaBytes = 0, kLoads = 2;
};

__device__ __forceinline__ float f16_lo(uint32_t v) { return f16_bits_to_f32((uint16_t)(v & 0xffffu)); }
__device__ __forceinline__ float f16_hi(uint32_t v) { return f16_bits_to_f32((uint16_t)(v >> 16)); }

// Eight int4 codes (k = 8G + 0..7 in nibble order) -> bf16 (128 + q) in the
// slot order (i, i + 4): dword i holds nibble i in its low half and nibble
// i + 4 in its high half.  `mask` (0x000F000F) and `exp` (0x43004300) come in
// registers: a VOP3 instruction on gfx950 takes no literal operand, so with
// literal masks each (a & mask) | exp becomes two instructions instead of one
// v_and_or_b32.
__device__ __forceinline__ bf16x8_t int4_octet_as_offset_bf16(uint32_t w, uint32_t mask, uint32_t exp) {
  return as_bf16x8(make_uint4((w & mask) | exp, ((w >> 4) & mask) | exp, ((w >> 8) & mask) | exp,
                              ((w >> 12) & mask) | exp));
}

// Eight int8 codes (k = 8G + 0..3 in lo, 4..7 in hi) -> bf16 (exact) in the
// slot order (i, i + 4).
__device__ __forceinline__ bf16x8_t int8_octet_as_bf16(uint32_t lo, uint32_t hi) {
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float a = (float)(int8_t)(lo >> (8 * i));
    const float b = (float)(int8_t)(hi >> (8 * i));
    o[i] = __builtin_amdgcn_perm(__float_as_uint(b), __float_as_uint(a), 0x07060302u);  // (a, b) upper halves
  }
  return as_bf16x8(make_uint4(o[0], o[1], o[2], o[3]));
}

template <Quant Q, Epi E>
__global__ __launch_bounds__(kGvThreads) void gemv_q_kernel(GemmParams p) {
  using U = GvUnit<Q>;
  extern __shared__ __attribute__((aligned(16))) uint8_t gv_lds[];
  const int M = p.M, N = p.N, K = p.K;
  const int n0 = blockIdx.x * 16;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, G = lane >> 4;
  const int units = K / kGvUnitK;
  const int nu = units > wave ? (units - wave + kGvWaves - 1) / kGvWaves : 0;  // this wave's units

  // LDS: code slots [kGvWaves][kGvDepth] | int4 scale/zero slots [kGvWaves][kGvDepth]
  //      | activations [K/8][M][16 B] | group sums [K/32][M] f32
  // (every direct-to-LDS destination is aligned to its own size)
  uint8_t* ring = gv_lds + wave * kGvDepth * U::kCodeBytes;
  uint8_t* meta = gv_lds + kGvWaves * kGvDepth * U::kCodeBytes + wave * kGvDepth * U::kMetaBytes;
  uint8_t* xl = gv_lds + kGvWaves * kGvDepth * (U::kCodeBytes + U::kMetaBytes);
  float* xs = reinterpret_cast<float*>(xl + (size_t)M * K * 2);

  // 1. Activations, as stored, into LDS: direct loads issued before the
  //    unit loads, so that waiting for them leaves the units in flight.
  constexpr int kOctPerThread = kGvMaxXBytes / 16 / kGvThreads;
  const int octets = M * K / 8;  // 16-byte octets of x, a multiple of 16
  const int oct_per_row = K / 8;
  const uint32_t xl_addr = lds_addr_of(xl);
#pragma unroll
  for (int i = 0; i < kOctPerThread; ++i) {
    const int q0 = wave * 64 + i * kGvThreads;  // octet of lane 0 in this load
    if (q0 < octets && q0 + lane < octets)
      lds_dma16(reinterpret_cast<const bf16_t*>(p.x) + (size_t)(q0 + lane) * 8,
                __builtin_amdgcn_readfirstlane(xl_addr + q0 * 16));
  }

  // 2. Unit loads.  Unit u, columns n0..n0+15: lane (row l16, chunk G) of the
  //    wave moves 16 bytes; slot layout [chunk][row][16 B].
  const size_t wpitch = Q == Quant::Int4 ? (size_t)K / 2 : (size_t)K;
  const uint8_t* wbase = reinterpret_cast<const uint8_t*>(p.w) + (size_t)(n0 + l16) * wpitch + G * 16;
  // int4 scales and zeros ([N][K/32] f16): lanes < 32 move the scales of row
  // lane/2, the others the zeros of row (lane-32)/2, two groups (4 bytes) each
  const size_t gpitch = (size_t)K / 32 * 2;
  const uint8_t* sz_base =
      Q == Quant::Int4 ? reinterpret_cast<const uint8_t*>(lane < 32 ? p.scales : p.zeros) +
                             (size_t)(n0 + ((lane & 31) >> 1)) * gpitch + (lane & 1) * 4
                       : nullptr;
  const uint32_t ring_addr = lds_addr_of(ring), meta_addr = lds_addr_of(meta);
  auto issue = [&](int i) {
    const int u = wave + i * kGvWaves;
    const uint32_t slot = ring_addr + (uint32_t)((i % kGvDepth) * U::kCodeBytes);
    if constexpr (Q == Quant::Int4) {
      lds_dma16(wbase + (size_t)u * 64, __builtin_amdgcn_readfirstlane(slot));
      lds_dma4(sz_base + (size_t)u * 8,
               __builtin_amdgcn_readfirstlane(meta_addr + (uint32_t)((i % kGvDepth) * U::kMetaBytes)));
    } else {
      lds_dma16(wbase + (size_t)u * 128, __builtin_amdgcn_readfirstlane(slot));
      lds_dma16(wbase + (size_t)u * 128 + 64, __builtin_amdgcn_readfirstlane(slot + 1024));
    }
  };
  const int pro = min(nu, kGvDepth);
  for (int i = 0; i < pro; ++i) issue(i);

  // 3. Activations rewritten in place in slot order ([K/8][M][16 B], bf16
  //    pairs (i, i + 4) of each octet), and the per-group sums.
  wait_stage<U::kLoads, kGvDepth>(pro);  // this wave's activation loads (older) have landed
  uint4 xr[kOctPerThread];
#pragma unroll
  for (int i = 0; i < kOctPerThread; ++i) {
    const int q = tid + i * kGvThreads;
    if (q < octets) xr[i] = *reinterpret_cast<const uint4*>(xl + (size_t)q * 16);
  }
  __syncthreads();  // every stored octet is in registers before any is overwritten
#pragma unroll
  for (int i = 0; i < kOctPerThread; ++i) {
    const int q = tid + i * kGvThreads;
    if (q < octets) {  // uniform over the 4 lanes of a group
      const int m = q / oct_per_row, o = q - m * oct_per_row;
      const uint4 v = xr[i];
      const uint4 e = make_uint4(__builtin_amdgcn_perm(v.z, v.x, 0x05040100u), __builtin_amdgcn_perm(v.z, v.x, 0x07060302u),
                                 __builtin_amdgcn_perm(v.w, v.y, 0x05040100u), __builtin_amdgcn_perm(v.w, v.y, 0x07060302u));
      *reinterpret_cast<uint4*>(xl + ((size_t)o * M + m) * 16) = e;
      const uint32_t d[4] = {v.x, v.y, v.z, v.w};
      float t = 0.0f;
#pragma unroll
      for (int j = 0; j < 4; ++j) t += __uint_as_float(d[j] << 16) + __uint_as_float(d[j] & 0xffff0000u);
      // the group's four octets sit on lanes 4a .. 4a+3 (quad_perm xor 1, then xor 2)
      t += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, t), 0xB1, 0xF, 0xF, false));
      t += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, t), 0x4E, 0xF, 0xF, false));
      if ((q & 3) == 0) xs[(o >> 2) * M + m] = t;
    }
  }
  __syncthreads();

  // 4. K loop.
  const int mc = min(l16, M - 1);  // A-operand row of this lane
  f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
  const f32x4_t zero4 = {0.0f, 0.0f, 0.0f, 0.0f};
  // nibble pair mask and the bf16 exponent of 128, as register values the
  // compiler cannot fold back into literals (see int4_octet_as_offset_bf16)
  uint32_t kMask, kExp;
  asm volatile("v_mov_b32 %0, 0x000F000F" : "=v"(kMask));
  asm volatile("v_mov_b32 %0, 0x43004300" : "=v"(kExp));
  for (int i = 0; i < nu; ++i) {
    wait_stage<U::kLoads, kGvDepth - 1>(min(nu - 1 - i, kGvDepth - 1));  // unit i has landed
    const int u = wave + i * kGvWaves;
    const uint8_t* slot = ring + (i % kGvDepth) * U::kCodeBytes;
    const uint8_t* mslot = meta + (i % kGvDepth) * U::kMetaBytes;
    bf16x8_t xa[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      xa[j] = as_bf16x8(*reinterpret_cast<const uint4*>(xl + ((size_t)(16 * u + 4 * j + G) * M + mc) * 16));
    if constexpr (Q == Quant::Int4) {
      const uint32_t* cw = reinterpret_cast<const uint32_t*>(slot + l16 * 16 + G * 4);
      const uint32_t c0 = cw[0], c1 = cw[64], c2 = cw[128], c3 = cw[192];
      const uint2 sv = *reinterpret_cast<const uint2*>(mslot + l16 * 8);
      const uint16_t zg = *reinterpret_cast<const uint16_t*>(mslot + 128 + l16 * 8 + G * 2);
      const uint16_t sg = *reinterpret_cast<const uint16_t*>(mslot + l16 * 8 + G * 2);
      const float xsum = xs[(4 * u + G) * M + mc];
      wait_lgkmcnt0();
      if (i + kGvDepth < nu) issue(i + kGvDepth);  // the slot's bytes are all in registers
      const f32x4_t v0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[0], int4_octet_as_offset_bf16(c0, kMask, kExp), zero4, 0, 0, 0);
      const f32x4_t v1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[1], int4_octet_as_offset_bf16(c1, kMask, kExp), zero4, 0, 0, 0);
      const f32x4_t v2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[2], int4_octet_as_offset_bf16(c2, kMask, kExp), zero4, 0, 0, 0);
      const f32x4_t v3 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[3], int4_octet_as_offset_bf16(c3, kMask, kExp), zero4, 0, 0, 0);
      const float negc = -f16_bits_to_f32(sg) * (128.0f + f16_bits_to_f32(zg));
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xsum, negc, acc, 0, 0, 0);
      const float s0 = f16_lo(sv.x), s1 = f16_hi(sv.x), s2 = f16_lo(sv.y), s3 = f16_hi(sv.y);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] = fmaf(s0, v0[r], fmaf(s1, v1[r], fmaf(s2, v2[r], fmaf(s3, v3[r], acc[r]))));
    } else {
      const uint2* cw = reinterpret_cast<const uint2*>(slot + (G >> 1) * 256 + l16 * 16 + (G & 1) * 8);
      const uint2 c0 = cw[0], c1 = cw[64], c2 = cw[128], c3 = cw[192];
      wait_lgkmcnt0();
      if (i + kGvDepth < nu) issue(i + kGvDepth);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[0], int8_octet_as_bf16(c0.x, c0.y), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[1], int8_octet_as_bf16(c1.x, c1.y), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[2], int8_octet_as_bf16(c2.x, c2.y), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[3], int8_octet_as_bf16(c3.x, c3.y), acc, 0, 0, 0);
    }
  }

  // 5. Wave partials -> LDS (each wave into its own ring: its loads have all
  //    landed and been read), then one thread per output adds them in wave order.
  *reinterpret_cast<f32x4_t*>(ring + lane * 16) = acc;
  __syncthreads();
  if (tid < 16 * kGvMaxRows) {
    const int m = tid >> 4, n = tid & 15;  // output (m, n0 + n) is register m % 4 of lane n + 16 (m / 4)
    if (m < M) {
      const int src = (n + 16 * (m >> 2)) * 16 + (m & 3) * 4;
      float v = 0.0f;
#pragma unroll
      for (int w = 0; w < kGvWaves; ++w) v += *reinterpret_cast<const float*>(gv_lds + w * kGvDepth * U::kCodeBytes + src);
      if constexpr (Q == Quant::Int8) v *= f16_bits_to_f32(reinterpret_cast<const uint16_t*>(p.scales)[n0 + n]);
      if constexpr (E != Epi::None) v += p.bias[n0 + n];
      if constexpr (E == Epi::BiasGelu) v = gelu_erf(v);
      if constexpr (E == Epi::BiasResidual) v += bf16_to_f32(reinterpret_cast<const bf16_t*>(p.residual)[(size_t)m * N + n0 + n]);
      reinterpret_cast<bf16_t*>(p.y)[(size_t)m * N + n0 + n] = f32_to_bf16(v);
    }
  }
}

template <Quant Q, Epi E>
hipError_t launch_gemv_typed(const GemmParams& p, hipStream_t s) {
  const size_t lds = gemv_lds_bytes(p);
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(gemv_q_kernel<Q, E>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((gemv_q_kernel<Q, E>), dim3(p.N / 16), dim3(kGvThreads), lds, s, p);
  return hipGetLastError();
}

template <Quant Q>
hipError_t launch_gemv_q(const GemmParams& p, hipStream_t s) {
  switch (p.epi) {
    case Epi::None: return launch_gemv_typed<Q, Epi::None>(p, s);
    case Epi::Bias: return launch_gemv_typed<Q, Epi::Bias>(p, s);
    case Epi::BiasGelu: return launch_gemv_typed<Q, Epi::BiasGelu>(p, s);
    case Epi::BiasResidual: return launch_gemv_typed<Q, Epi::BiasResidual>(p, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

size_t gemv_lds_bytes(const GemmParams& p) {
  const int slot = p.quant == Quant::Int4 ? GvUnit<Quant::Int4>::kCodeBytes + GvUnit<Quant::Int4>::kMetaBytes
                                          : GvUnit<Quant::Int8>::kCodeBytes + GvUnit<Quant::Int8>::kMetaBytes;
  return (size_t)kGvWaves * kGvDepth * slot + (size_t)p.M * p.K * 2 + (size_t)p.M * (p.K / 32) * 4;
}

bool gemv_supported(const GemmParams& p) {
  auto a4 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 3) == 0; };
  return (p.quant == Quant::Int4 || p.quant == Quant::Int8) && p.dtype == DType::BF16 && p.m_dev == nullptr &&
         p.x_head_rows == 0 && !p.x_stats && !p.res_stats && !p.y_stats && p.M >= 1 && p.M <= kGvMaxRows &&
         p.N % 16 == 0 && p.K % kGvUnitK == 0 && (size_t)p.M * p.K * 2 <= (size_t)kGvMaxXBytes &&
         (p.quant == Quant::Int8 || (a4(p.scales) && a4(p.zeros)));
}

hipError_t launch_gemv(const GemmParams& p, hipStream_t s) {
  if (!gemv_supported(p)) return hipErrorInvalidValue;
  return p.quant == Quant::Int4 ? launch_gemv_q<Quant::Int4>(p, s) : launch_gemv_q<Quant::Int8>(p, s);
}

}  // namespace rlx
