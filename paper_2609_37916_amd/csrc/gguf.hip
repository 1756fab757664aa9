// GGUF weight blocks -> the dequantising matmul's own layouts (the llama.cpp
// scheme set of Op::DequantMatMul, Section VI).
//
// A GGUF tensor row is a run of 32-weight blocks: Q4_0 (18 bytes: f16 d,
// 16 bytes of nibbles, W = (q - 8) d), Q4_1 (20 bytes: f16 d, f16 m, nibbles,
// W = q d + m), Q8_0 (34 bytes: f16 d, 32 int8, W = q d); in a 4-bit block
// element j < 16 is the low and element j + 16 the high nibble of byte j.
// Blocks are 2-byte aligned at best, which suits neither 16-byte loads nor
// the MFMA operand layouts, so weights are re-laid out once, at load time,
// into layouts whose values are the same numbers:
//   Q4_0 -> Int4  (codes two per byte, k = 2j low nibble; s = d, z = 8)
//   Q4_1 -> Int4M (same codes; s = d, m = m)
//   Q8_0 -> Int8G (int8 codes; s = d)
// One thread per block: f16 fields and code bytes are read as 16-bit words.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace rlx {
namespace {

constexpr int kQ4_0 = 2, kQ4_1 = 3, kQ8_0 = 8;  // GGUF tensor type ids

template <int TYPE>
__global__ __launch_bounds__(256) void gguf_repack_kernel(const uint16_t* blocks, int N, int K, uint8_t* codes,
                                                          uint16_t* scales, uint16_t* zeros) {
  constexpr int kHalves = TYPE == kQ4_0 ? 9 : (TYPE == kQ4_1 ? 10 : 17);  // block size / 2
  const int nb = K / 32;
  const size_t total = (size_t)N * nb;
  for (size_t b = (size_t)blockIdx.x * blockDim.x + threadIdx.x; b < total; b += (size_t)gridDim.x * blockDim.x) {
    const uint16_t* src = blocks + b * kHalves;
    uint16_t h[kHalves];
#pragma unroll
    for (int i = 0; i < kHalves; ++i) h[i] = src[i];
    scales[b] = h[0];
    if constexpr (TYPE == kQ8_0) {
      uint32_t w[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) w[i] = (uint32_t)h[1 + 2 * i] | ((uint32_t)h[2 + 2 * i] << 16);
      uint4* dst = reinterpret_cast<uint4*>(codes + b * 32);  // row n, block j: n * K + 32 j
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    } else {
      constexpr int off = TYPE == kQ4_0 ? 1 : 2;  // first half-word of the nibbles
      zeros[b] = TYPE == kQ4_0 ? (uint16_t)0x4800u : h[1];  // f16 8.0, or the block's m
      uint8_t qs[16];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        qs[2 * i] = (uint8_t)(h[off + i] & 0xffu);
        qs[2 * i + 1] = (uint8_t)(h[off + i] >> 8);
      }
      // our byte j holds elements 2j (low) and 2j+1 (high)
      uint8_t o[16];
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = (uint8_t)((qs[2 * j] & 0xf) | ((qs[2 * j + 1] & 0xf) << 4));
#pragma unroll
      for (int j = 8; j < 16; ++j) o[j] = (uint8_t)((qs[2 * j - 16] >> 4) | (qs[2 * j - 15] & 0xf0));
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        w[i] = (uint32_t)o[4 * i] | ((uint32_t)o[4 * i + 1] << 8) | ((uint32_t)o[4 * i + 2] << 16) |
               ((uint32_t)o[4 * i + 3] << 24);
      *reinterpret_cast<uint4*>(codes + b * 16) = make_uint4(w[0], w[1], w[2], w[3]);  // n * K/2 + 16 j
    }
  }
}

template <int TYPE>
hipError_t launch_repack(const void* blocks, int N, int K, void* codes, void* scales, void* zeros, hipStream_t s) {
  const size_t total = (size_t)N * (K / 32);
  const int grid = (int)std::min<size_t>((total + 255) / 256, 4096);
  RLX_LOG_LAUNCH("gguf_repack_kernel", dim3(grid), dim3(256), 0, "type=%d", (int)TYPE);
  hipLaunchKernelGGL(gguf_repack_kernel<TYPE>, dim3(grid), dim3(256), 0, s, reinterpret_cast<const uint16_t*>(blocks),
                     N, K, reinterpret_cast<uint8_t*>(codes), reinterpret_cast<uint16_t*>(scales),
                     reinterpret_cast<uint16_t*>(zeros));
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gguf_repack(const void* blocks, int type, int N, int K, void* codes, void* scales, void* zeros,
                              hipStream_t s) {
  if (N <= 0) return hipSuccess;
  switch (type) {
    case kQ4_0: return launch_repack<kQ4_0>(blocks, N, K, codes, scales, zeros, s);
    case kQ4_1: return launch_repack<kQ4_1>(blocks, N, K, codes, scales, zeros, s);
    case kQ8_0: return launch_repack<kQ8_0>(blocks, N, K, codes, scales, zeros, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace rlx
