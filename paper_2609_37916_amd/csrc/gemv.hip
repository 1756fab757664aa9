// Dequantising matmul for a few activation rows (the GEMV regime of
// Op::DequantMatMul, Section VI; Linear block, Section III-A):
//
//   y[m, n] = epi( sum_k x[m, k] W[n, k] ),   1 <= M <= 16 bf16 rows,
//
// with W in the int8 per-channel, int4 group-32 zero-point, int8 group-32,
// int8 group-16 or int4 group-32 min layout (the last three also hold GGUF
// Q8_0, Q6_K and Q4_1 / Q4_K weights).
// With so few rows the product reads every weight byte once and does little
// arithmetic per byte: it is bound by HBM bandwidth and by the vector-ALU
// work of unpacking the codes, not by the matrix cores.
//
//  * Output columns go in tiles of 16.  Each block takes a contiguous run of
//    tiles (about two blocks per CU, so the activations are staged once per
//    block and no second wave of blocks leaves a tail).  Within a tile the 8
//    waves split K in 128-k units (unit u goes to wave u mod 8); at the end of
//    the tile the 8 partial 16 x 16 tiles are added in LDS in wave order
//    (deterministic) and the epilogue is applied.
//  * Each wave streams its (tile, unit) items through a private ring of LDS
//    slots with direct-to-LDS loads, two to four items in flight (per
//    layout, measured) across tile boundaries; the only barrier is the one
//    per tile that hands the wave partials to the epilogue (double-buffered).
//    A unit's 16 weight rows land group-major ([16-byte chunk][row][16 B]):
//    lane (n, G) then reads the 4 (int4) or 8 (int8) bytes of k-octet G of
//    each group with conflict-free ds_read2.
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
//    each (q - z) s to bf16).  int4 min (W = q s + m) is the same with
//    (m - 128 s) X in place of -s (128 + z) X.
//  * int8 per-channel: codes convert exactly to bf16 and one accumulator
//    takes every group; the per-channel scale multiplies the fp32 sum in the
//    epilogue, as in the tiled path.  int8 group: each group's product is
//    scaled by its s with four FMAs a lane, as for int4.  int8 group-16: a
//    32-k instruction would add two groups of different scale, so each group
//    of 32 takes two instructions, the lanes of the other half (k-octets 2, 3
//    for the first, 0, 1 for the second) supplying zero codes; each product is
//    scaled by its own s, as for group 32.
#include "common.hpp"
#include "kernels.hpp"

namespace rlx {
namespace {

constexpr int kGvWaves = 8;
constexpr int kGvThreads = kGvWaves * 64;
constexpr int kGvUnitK = 128;       // k per unit (four 32-k groups)
constexpr int kGvMaxRows = 16;
constexpr int kGvMaxXBytes = 64 * 1024;  // activations staged in LDS (bf16)

template <Quant Q>
struct GvUnit;
template <>
struct GvUnit<Quant::Int4> {
  // codes: 16 rows x 64 bytes; meta: scales then zeros, 16 rows x 4 f16 each;
  // kDepth items in flight per wave (measured on the 14336 x 4096 product:
  // 2 in flight 12.0 us, 3 13.3 us, 4 14.0 us)
  static constexpr int kCodeBytes = 1024, kMetaBytes = 256, kLoads = 2, kDepth = 2;
};
template <>
struct GvUnit<Quant::Int4M> : GvUnit<Quant::Int4> {};  // zeros hold the mins
template <>
struct GvUnit<Quant::Int8G> {
  // codes: 16 rows x 128 bytes; meta: 16 rows x 4 f16 scales (then a copy)
  static constexpr int kCodeBytes = 2048, kMetaBytes = 256, kLoads = 3, kDepth = 3;
};
template <>
struct GvUnit<Quant::Int8G16> {
  // codes: 16 rows x 128 bytes; meta: 16 rows x 8 f16 scales
  static constexpr int kCodeBytes = 2048, kMetaBytes = 256, kLoads = 3, kDepth = 3;
};
template <>
struct GvUnit<Quant::Int8> {
  // (2 in flight 14.2 us, 3 14.0 us, 4 13.6 us)
  static constexpr int kCodeBytes = 2048, kMetaBytes = 0, kLoads = 2, kDepth = 4;
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

// Epilogue operands of a block's run of tpb tiles in LDS (byte offsets);
// every part is 256-byte aligned, the whole a multiple of 1 KB.
struct GvEpiLayout {
  int bias, scale, res, res_pitch, bytes;
};
__host__ __device__ constexpr int gv_round(int v, int a) { return (v + a - 1) / a * a; }
// (residual rows of y's element size: 2 bytes, or 4 for an f32 output)
__host__ __device__ inline GvEpiLayout gv_epi_layout(Quant q, Epi e, int M, int tpb, bool y_f32) {
  GvEpiLayout l{};
  int off = 0;
  l.bias = off;
  if (e != Epi::None) off += gv_round(tpb * 16 * 4, 256);
  l.scale = off;
  if (q == Quant::Int8) off += gv_round(tpb * 16 * 2, 256);
  l.res = off;
  l.res_pitch = gv_round(tpb * 16 * (y_f32 ? 4 : 2), 256);
  if (e == Epi::BiasResidual) off += M * l.res_pitch;
  l.bytes = gv_round(off, 1024);
  return l;
}

template <Quant Q, Epi E>
__global__ __launch_bounds__(kGvThreads) void gemv_q_kernel(GemmParams p) {
  using U = GvUnit<Q>;
  extern __shared__ __attribute__((aligned(16))) uint8_t gv_lds[];
  const int M = p.M, N = p.N, K = p.K;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, G = lane >> 4;
  const int units = K / kGvUnitK;
  const int nu = units > wave ? (units - wave + kGvWaves - 1) / kGvWaves : 0;  // this wave's units per tile
  // this block's tiles of 16 columns: t0 .. t0 + nt - 1
  const int tiles = N / 16;
  const int tpb = (tiles + gridDim.x - 1) / gridDim.x;
  const int t0 = blockIdx.x * tpb;
  const int nt = max(0, min(tiles - t0, tpb));
  const int items = nt * nu;  // (tile, unit) items of this wave, tile-major

  // LDS: code slots [kGvWaves][kDepth] | int4 scale/zero slots [kGvWaves][kDepth]
  //      | wave partials [2][kGvWaves][64 lanes][4] f32 | epilogue operands of
  //      the block's tiles (GvEpiLayout) | activations [K/8][M][16 B]
  //      | group sums [K/32][M] f32   (direct-to-LDS destinations 256-byte aligned)
  uint8_t* ring = gv_lds + wave * U::kDepth * U::kCodeBytes;
  uint8_t* meta = gv_lds + kGvWaves * U::kDepth * U::kCodeBytes + wave * U::kDepth * U::kMetaBytes;
  uint8_t* red = gv_lds + kGvWaves * U::kDepth * (U::kCodeBytes + U::kMetaBytes);
  const GvEpiLayout el = gv_epi_layout(Q, E, M, tpb, p.y_f32);
  uint8_t* epi = red + 2 * kGvWaves * 1024;
  uint8_t* xl = epi + el.bytes;
  float* xs = reinterpret_cast<float*>(xl + (size_t)M * K * 2);

  // 1. Activations, as stored, into LDS.
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

  // Epilogue operands of the block's tiles (bias, int8 scales, residual
  // rows), 4 bytes a lane: each wave moves the rows m = wave mod 8 of the
  // residual; wave 0 the bias, wave 1 the scales.
  const int ncol = nt * 16;  // this block's columns, from column 16 t0
  auto dma_run = [&](const void* src, uint8_t* dst, int dwords) {
    for (int j = 0; j * 64 < dwords; ++j)
      if (j * 64 + lane < dwords)
        lds_dma4(reinterpret_cast<const uint32_t*>(src) + j * 64 + lane,
                 __builtin_amdgcn_readfirstlane(lds_addr_of(dst) + j * 256));
  };
  if constexpr (E != Epi::None)
    if (wave == 0) dma_run(p.bias + (size_t)t0 * 16, epi + el.bias, ncol);
  if constexpr (Q == Quant::Int8)
    if (wave == 1) dma_run(reinterpret_cast<const uint16_t*>(p.scales) + (size_t)t0 * 16, epi + el.scale, ncol / 2);
  if constexpr (E == Epi::BiasResidual)
    for (int m = wave; m < M; m += kGvWaves) {
      if (p.y_f32)
        dma_run(reinterpret_cast<const float*>(p.residual) + (size_t)m * N + (size_t)t0 * 16,
                epi + el.res + m * el.res_pitch, ncol);
      else
        dma_run(reinterpret_cast<const bf16_t*>(p.residual) + (size_t)m * N + (size_t)t0 * 16,
                epi + el.res + m * el.res_pitch, ncol / 2);
    }

  // 2. Item loads.  Item (tile t, unit u): lane (row l16, chunk G) of the
  //    wave moves 16 bytes of row 16 t + l16; slot layout [chunk][row][16 B].
  const size_t wpitch = quant_int4(Q) ? (size_t)K / 2 : (size_t)K;
  const uint8_t* wlane = reinterpret_cast<const uint8_t*>(p.w) + (size_t)l16 * wpitch + G * 16;
  // int4 scales and zeros ([N][K/32] f16): lanes < 32 move the scales of row
  // lane/2, the others the zeros of row (lane-32)/2, two groups (4 bytes) each
  // (int8 group scales: every lane moves scales, lanes >= 32 a second copy;
  // group 16 ([N][K/16] f16): lane moves two of the eight scales of row lane/4)
  constexpr bool kG16 = Q == Quant::Int8G16;
  const size_t gpitch = (size_t)K / (kG16 ? 16 : 32) * 2;
  const uint8_t* mlane =
      U::kMetaBytes == 0 ? nullptr
      : kG16 ? reinterpret_cast<const uint8_t*>(p.scales) + (size_t)(lane >> 2) * gpitch + (lane & 3) * 4
             : reinterpret_cast<const uint8_t*>(lane < 32 || Q == Quant::Int8G ? p.scales : p.zeros) +
                   (size_t)((lane & 31) >> 1) * gpitch + (lane & 1) * 4;
  const uint32_t ring_addr = lds_addr_of(ring), meta_addr = lds_addr_of(meta);
  auto issue = [&](int i) {
    const int tt = i / nu, u = wave + (i - tt * nu) * kGvWaves;
    const size_t row0 = (size_t)(t0 + tt) * 16;
    const uint32_t slot = ring_addr + (uint32_t)((i % U::kDepth) * U::kCodeBytes);
    if constexpr (quant_int4(Q)) {
      lds_dma16(wlane + row0 * wpitch + (size_t)u * 64, __builtin_amdgcn_readfirstlane(slot));
    } else {
      lds_dma16(wlane + row0 * wpitch + (size_t)u * 128, __builtin_amdgcn_readfirstlane(slot));
      lds_dma16(wlane + row0 * wpitch + (size_t)u * 128 + 64, __builtin_amdgcn_readfirstlane(slot + 1024));
    }
    if constexpr (U::kMetaBytes > 0)
      lds_dma4(mlane + row0 * gpitch + (size_t)u * (kG16 ? 16 : 8),
               __builtin_amdgcn_readfirstlane(meta_addr + (uint32_t)((i % U::kDepth) * U::kMetaBytes)));
  };
  // The activations are waited for before any item load goes out.  (Issuing
  // the first items before that wait measured the same within 0.5 us: the
  // activations then queue behind other blocks' weight bytes instead.)
  wait_vmcnt<0>();
  const int pro = min(items, U::kDepth);
  for (int i = 0; i < pro; ++i) issue(i);

  // 3. Activations rewritten in place in slot order ([K/8][M][16 B], bf16
  //    pairs (i, i + 4) of each octet), and the per-group sums.
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

  // 4. Tiles: K loop per tile, then the wave partials to the epilogue.
  const int mc = min(l16, M - 1);  // A-operand row of this lane
  const f32x4_t zero4 = {0.0f, 0.0f, 0.0f, 0.0f};
  // nibble pair mask and the bf16 exponent of 128, as register values the
  // compiler cannot fold back into literals (see int4_octet_as_offset_bf16)
  uint32_t kMask, kExp;
  asm volatile("v_mov_b32 %0, 0x000F000F" : "=v"(kMask));
  asm volatile("v_mov_b32 %0, 0x43004300" : "=v"(kExp));
  for (int tt = 0; tt < nt; ++tt) {
    f32x4_t acc = zero4;
    for (int j = 0; j < nu; ++j) {
      const int i = tt * nu + j;
      wait_stage<U::kLoads, U::kDepth - 1>(min(items - 1 - i, U::kDepth - 1));  // item i has landed
      const int u = wave + j * kGvWaves;
      const uint8_t* slot = ring + (i % U::kDepth) * U::kCodeBytes;
      const uint8_t* mslot = meta + (i % U::kDepth) * U::kMetaBytes;
      bf16x8_t xa[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        xa[q] = as_bf16x8(*reinterpret_cast<const uint4*>(xl + ((size_t)(16 * u + 4 * q + G) * M + mc) * 16));
      if constexpr (quant_int4(Q)) {
        const uint32_t* cw = reinterpret_cast<const uint32_t*>(slot + l16 * 16 + G * 4);
        const uint32_t c0 = cw[0], c1 = cw[64], c2 = cw[128], c3 = cw[192];
        const uint2 sv = *reinterpret_cast<const uint2*>(mslot + l16 * 8);
        const uint16_t zg = *reinterpret_cast<const uint16_t*>(mslot + 128 + l16 * 8 + G * 2);
        const uint16_t sg = *reinterpret_cast<const uint16_t*>(mslot + l16 * 8 + G * 2);
        const float xsum = xs[(4 * u + G) * M + mc];
        wait_lgkmcnt0();
        if (i + U::kDepth < items) issue(i + U::kDepth);  // the slot's bytes are all in registers
        const f32x4_t v0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[0], int4_octet_as_offset_bf16(c0, kMask, kExp), zero4, 0, 0, 0);
        const f32x4_t v1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[1], int4_octet_as_offset_bf16(c1, kMask, kExp), zero4, 0, 0, 0);
        const f32x4_t v2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[2], int4_octet_as_offset_bf16(c2, kMask, kExp), zero4, 0, 0, 0);
        const f32x4_t v3 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[3], int4_octet_as_offset_bf16(c3, kMask, kExp), zero4, 0, 0, 0);
        // int4: s V - s (128 + z) X;  int4 min (zg holds m): s V + (m - 128 s) X
        const float negc = Q == Quant::Int4 ? -f16_bits_to_f32(sg) * (128.0f + f16_bits_to_f32(zg))
                                            : fmaf(-128.0f, f16_bits_to_f32(sg), f16_bits_to_f32(zg));
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xsum, negc, acc, 0, 0, 0);
        const float s0 = f16_lo(sv.x), s1 = f16_hi(sv.x), s2 = f16_lo(sv.y), s3 = f16_hi(sv.y);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] = fmaf(s0, v0[r], fmaf(s1, v1[r], fmaf(s2, v2[r], fmaf(s3, v3[r], acc[r]))));
      } else if constexpr (Q == Quant::Int8G) {
        const uint2* cw = reinterpret_cast<const uint2*>(slot + (G >> 1) * 256 + l16 * 16 + (G & 1) * 8);
        const uint2 c0 = cw[0], c1 = cw[64], c2 = cw[128], c3 = cw[192];
        const uint2 sv = *reinterpret_cast<const uint2*>(mslot + l16 * 8);
        wait_lgkmcnt0();
        if (i + U::kDepth < items) issue(i + U::kDepth);
        const f32x4_t v0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[0], int8_octet_as_bf16(c0.x, c0.y), zero4, 0, 0, 0);
        const f32x4_t v1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[1], int8_octet_as_bf16(c1.x, c1.y), zero4, 0, 0, 0);
        const f32x4_t v2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[2], int8_octet_as_bf16(c2.x, c2.y), zero4, 0, 0, 0);
        const f32x4_t v3 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[3], int8_octet_as_bf16(c3.x, c3.y), zero4, 0, 0, 0);
        const float s0 = f16_lo(sv.x), s1 = f16_hi(sv.x), s2 = f16_lo(sv.y), s3 = f16_hi(sv.y);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] = fmaf(s0, v0[r], fmaf(s1, v1[r], fmaf(s2, v2[r], fmaf(s3, v3[r], acc[r]))));
      } else if constexpr (Q == Quant::Int8G16) {
        const uint2* cw = reinterpret_cast<const uint2*>(slot + (G >> 1) * 256 + l16 * 16 + (G & 1) * 8);
        const uint2 c0 = cw[0], c1 = cw[64], c2 = cw[128], c3 = cw[192];
        const uint4 sv = *reinterpret_cast<const uint4*>(mslot + l16 * 16);
        wait_lgkmcnt0();
        if (i + U::kDepth < items) issue(i + U::kDepth);
        // group 2q (k 32q .. 32q + 15) is k-octets 0, 1 of instruction q, group 2q + 1 octets 2, 3
        const bool first = G < 2;
        const bf16x8_t zb = as_bf16x8(make_uint4(0u, 0u, 0u, 0u));
        const uint2 cc[4] = {c0, c1, c2, c3};
        const uint32_t sw[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const bf16x8_t b = int8_octet_as_bf16(cc[q].x, cc[q].y);
          const f32x4_t va = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[q], first ? b : zb, zero4, 0, 0, 0);
          const f32x4_t vb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[q], first ? zb : b, zero4, 0, 0, 0);
          const float sa = f16_lo(sw[q]), sb = f16_hi(sw[q]);
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[r] = fmaf(sa, va[r], fmaf(sb, vb[r], acc[r]));
        }
      } else {
        const uint2* cw = reinterpret_cast<const uint2*>(slot + (G >> 1) * 256 + l16 * 16 + (G & 1) * 8);
        const uint2 c0 = cw[0], c1 = cw[64], c2 = cw[128], c3 = cw[192];
        wait_lgkmcnt0();
        if (i + U::kDepth < items) issue(i + U::kDepth);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[0], int8_octet_as_bf16(c0.x, c0.y), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[1], int8_octet_as_bf16(c1.x, c1.y), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[2], int8_octet_as_bf16(c2.x, c2.y), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[3], int8_octet_as_bf16(c3.x, c3.y), acc, 0, 0, 0);
      }
    }
    // The partials of tile tt go to buffer tt % 2: the epilogue of tile tt - 2,
    // the last reader of that buffer, ran before the barrier of tile tt - 1.
    uint8_t* rb = red + (tt & 1) * kGvWaves * 1024;
    *reinterpret_cast<f32x4_t*>(rb + wave * 1024 + lane * 16) = acc;
    __syncthreads();
    if (tid < 16 * kGvMaxRows) {
      const int m = tid >> 4, n = (t0 + tt) * 16 + (tid & 15);
      if (m < M) {  // output (m, n) is register m % 4 of lane n % 16 + 16 (m / 4)
        const int src = ((tid & 15) + 16 * (m >> 2)) * 16 + (m & 3) * 4;
        float v = 0.0f;
#pragma unroll
        for (int w = 0; w < kGvWaves; ++w) v += *reinterpret_cast<const float*>(rb + w * 1024 + src);
        const int c = tt * 16 + (tid & 15);  // column within the block's run
        if constexpr (Q == Quant::Int8) v *= f16_bits_to_f32(reinterpret_cast<const uint16_t*>(epi + el.scale)[c]);
        if constexpr (E != Epi::None) v += reinterpret_cast<const float*>(epi + el.bias)[c];
        if constexpr (E == Epi::BiasGelu) v = gelu_erf(v);
        if constexpr (E == Epi::BiasResidual)
          v += p.y_f32 ? reinterpret_cast<const float*>(epi + el.res + m * el.res_pitch)[c]
                       : bf16_to_f32(reinterpret_cast<const bf16_t*>(epi + el.res + m * el.res_pitch)[c]);
        if (p.y_f32)
          reinterpret_cast<float*>(p.y)[(size_t)m * N + n] = v;
        else
          reinterpret_cast<bf16_t*>(p.y)[(size_t)m * N + n] = f32_to_bf16(v);
      }
    }
  }
}

// Compute units of the current device (cached per device).
int device_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

struct GvPlan {
  int grid, tpb;
  size_t lds;
};

// Up to two blocks per CU (as many as the LDS allows), each with an equal run
// of tpb 16-column tiles; the LDS holds the rings, the wave partials, the
// run's epilogue operands and the activations.
GvPlan gemv_plan(const GemmParams& p) {
  using U4 = GvUnit<Quant::Int4>;
  using U8 = GvUnit<Quant::Int8>;
  using U8G = GvUnit<Quant::Int8G>;
  using U8G16 = GvUnit<Quant::Int8G16>;
  const int ring = quant_int4(p.quant)            ? U4::kDepth * (U4::kCodeBytes + U4::kMetaBytes)
                   : p.quant == Quant::Int8G     ? U8G::kDepth * (U8G::kCodeBytes + U8G::kMetaBytes)
                   : p.quant == Quant::Int8G16   ? U8G16::kDepth * (U8G16::kCodeBytes + U8G16::kMetaBytes)
                                                 : U8::kDepth * (U8::kCodeBytes + U8::kMetaBytes);
  const size_t base = (size_t)kGvWaves * ring + 2 * kGvWaves * 1024 + (size_t)p.M * p.K * 2 +
                      (size_t)p.M * (p.K / 32) * 4;
  const int tiles = p.N / 16;
  GvPlan g{};
  for (int per_cu = 2; per_cu >= 1; --per_cu) {
    g.tpb = (tiles + device_cus() * per_cu - 1) / (device_cus() * per_cu);
    g.lds = base + gv_epi_layout(p.quant, p.epi, p.M, g.tpb, p.y_f32).bytes;
    if (g.lds * per_cu <= 160 * 1024) break;
  }
  g.grid = (tiles + g.tpb - 1) / g.tpb;
  return g;
}

template <Quant Q, Epi E>
hipError_t launch_gemv_typed(const GemmParams& p, hipStream_t s) {
  const GvPlan g = gemv_plan(p);
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(gemv_q_kernel<Q, E>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  if (attr != hipSuccess) return attr;
  RLX_LOG_LAUNCH("gemv_q_kernel", dim3(g.grid), dim3(kGvThreads), g.lds, "few-row %s epi=%s M=%d N=%d K=%d",
                 quant_name(Q), epi_name(E), p.M, p.N, p.K);
  hipLaunchKernelGGL((gemv_q_kernel<Q, E>), dim3(g.grid), dim3(kGvThreads), g.lds, s, p);
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

bool gemv_supported(const GemmParams& p) {
  auto a4 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 3) == 0; };
  return p.quant != Quant::None && p.dtype == DType::BF16 && p.m_dev == nullptr &&
         p.x_head_rows == 0 && !p.x_stats && !p.res_stats && !p.y_stats && p.M >= 1 && p.M <= kGvMaxRows &&
         p.N % 16 == 0 && p.K % kGvUnitK == 0 && (size_t)p.M * p.K * 2 <= (size_t)kGvMaxXBytes &&
         a4(p.scales) && (!quant_int4(p.quant) || a4(p.zeros)) && gemv_plan(p).lds <= 160 * 1024;
}

hipError_t launch_gemv(const GemmParams& p, hipStream_t s) {
  if (!gemv_supported(p)) return hipErrorInvalidValue;
  switch (p.quant) {
    case Quant::Int4: return launch_gemv_q<Quant::Int4>(p, s);
    case Quant::Int4M: return launch_gemv_q<Quant::Int4M>(p, s);
    case Quant::Int8: return launch_gemv_q<Quant::Int8>(p, s);
    case Quant::Int8G: return launch_gemv_q<Quant::Int8G>(p, s);
    case Quant::Int8G16: return launch_gemv_q<Quant::Int8G16>(p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace rlx
