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
//
// K-quants come in 256-weight super-blocks with 6-bit (Q4_K) or 8-bit (Q6_K)
// sub-block scales under an f16 super-block scale:
//   Q4_K -> Int4M   (144 bytes: f16 d, f16 dmin, 12 bytes of 6-bit sub-block
//                    scales and mins, four runs of 32 nibble bytes;
//                    s = f16(d sc_j), m = f16(0 - dmin mn_j) per 32 weights)
//   Q6_K -> Int8G16 (210 bytes: 128 bytes of low nibbles, 64 of high bit
//                    pairs, 16 int8 scales, f16 d; codes q - 32 as int8,
//                    s = f16(d sc_i) per 16 weights)
// d sc_j and dmin mn_j are exact in fp32 (at most 17 and 19 significant
// bits) and are rounded once to f16 (nearest even), the internal layouts'
// scale type: the repacked weights are within 2^-11 (|s q| + |m|) of the
// format's values.  The composed values must be finite in f16.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace rlx {
namespace {

constexpr int kQ4_0 = 2, kQ4_1 = 3, kQ8_0 = 8, kQ4_K = 12, kQ6_K = 14;  // GGUF tensor type ids

__device__ __forceinline__ float f16v(uint16_t h) { return f16_bits_to_f32(h); }
__device__ __forceinline__ uint16_t f16_rne(float x) { return __builtin_bit_cast(uint16_t, (_Float16)x); }

// One thread per Q4_K super-block (72 half-words): codes to two per byte,
// k = 2j low nibble (128 bytes), eight f16 scales and mins.
__global__ __launch_bounds__(256) void q4_k_repack_kernel(const uint16_t* blocks, size_t total, uint8_t* codes,
                                                          uint16_t* scales, uint16_t* mins) {
  for (size_t b = (size_t)blockIdx.x * blockDim.x + threadIdx.x; b < total; b += (size_t)gridDim.x * blockDim.x) {
    const uint16_t* src = blocks + b * 72;
    const float d = f16v(src[0]), dmin = f16v(src[1]);
    uint8_t S[12];
#pragma unroll
    for (int i = 0; i < 6; ++i) {
      S[2 * i] = (uint8_t)(src[2 + i] & 0xffu);
      S[2 * i + 1] = (uint8_t)(src[2 + i] >> 8);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int sc = j < 4 ? (S[j] & 63) : ((S[j + 4] & 15) | ((S[j - 4] >> 6) << 4));
      const int mn = j < 4 ? (S[j + 4] & 63) : ((S[j + 4] >> 4) | ((S[j] >> 6) << 4));
      scales[b * 8 + j] = f16_rne(d * (float)sc);
      mins[b * 8 + j] = f16_rne(0.0f - dmin * (float)mn);  // a zero min is +0
    }
    // run c (weights 64c .. 64c+63): byte 32c + l holds weight 64c + l (low)
    // and 64c + 32 + l (high); output byte 32c + i holds weights 64c + 2i, 2i+1
    for (int c = 0; c < 4; ++c) {
      uint8_t qs[32];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const uint16_t h = src[8 + 16 * c + i];
        qs[2 * i] = (uint8_t)(h & 0xffu);
        qs[2 * i + 1] = (uint8_t)(h >> 8);
      }
      uint32_t w[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        uint32_t v = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int o = 4 * i + e;  // output byte: weights 2o, 2o + 1 of the run
          const int w0 = 2 * o, w1 = 2 * o + 1;
          const uint32_t n0 = w0 < 32 ? (qs[w0] & 15u) : (qs[w0 - 32] >> 4);
          const uint32_t n1 = w1 < 32 ? (qs[w1] & 15u) : (qs[w1 - 32] >> 4);
          v |= (n0 | (n1 << 4)) << (8 * e);
        }
        w[i] = v;
      }
      uint4* dst = reinterpret_cast<uint4*>(codes + b * 128 + 32 * c);
      dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
      dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    }
  }
}

// One thread per Q6_K super-block (105 half-words): int8 codes q - 32 in
// weight order (256 bytes) and sixteen f16 scales.
__global__ __launch_bounds__(256) void q6_k_repack_kernel(const uint16_t* blocks, size_t total, uint8_t* codes,
                                                          uint16_t* scales) {
  for (size_t b = (size_t)blockIdx.x * blockDim.x + threadIdx.x; b < total; b += (size_t)gridDim.x * blockDim.x) {
    const uint16_t* src = blocks + b * 105;
    const float d = f16v(src[104]);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint16_t h = src[96 + i];
      scales[b * 16 + 2 * i] = f16_rne(d * (float)(int8_t)(h & 0xffu));
      scales[b * 16 + 2 * i + 1] = f16_rne(d * (float)(int8_t)(h >> 8));
    }
    auto byte_at = [&](int o) -> uint32_t { return (src[o >> 1] >> (8 * (o & 1))) & 0xffu; };
    for (int half = 0; half < 2; ++half) {
      for (int quarter = 0; quarter < 4; ++quarter) {
        uint32_t w[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          uint32_t v = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int l = 4 * i + e;
            const uint32_t lo_byte = byte_at(64 * half + l + ((quarter & 1) ? 32 : 0));
            const uint32_t lo = quarter < 2 ? (lo_byte & 15u) : (lo_byte >> 4);
            const uint32_t hi = (byte_at(128 + 32 * half + l) >> (2 * quarter)) & 3u;
            v |= ((uint32_t)(uint8_t)(int8_t)((int)(lo | (hi << 4)) - 32)) << (8 * e);
          }
          w[i] = v;
        }
        uint4* dst = reinterpret_cast<uint4*>(codes + b * 256 + 128 * half + 32 * quarter);
        dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
        dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
      }
    }
  }
}

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
  if (type == kQ4_K || type == kQ6_K) {
    if (K % 256 != 0) return hipErrorInvalidValue;
    const size_t total = (size_t)N * (K / 256);
    const int grid = (int)std::min<size_t>((total + 255) / 256, 4096);
    RLX_LOG_LAUNCH(type == kQ4_K ? "q4_k_repack_kernel" : "q6_k_repack_kernel", dim3(grid), dim3(256), 0,
                   "N=%d K=%d", N, K);
    if (type == kQ4_K)
      hipLaunchKernelGGL(q4_k_repack_kernel, dim3(grid), dim3(256), 0, s, reinterpret_cast<const uint16_t*>(blocks),
                         total, reinterpret_cast<uint8_t*>(codes), reinterpret_cast<uint16_t*>(scales),
                         reinterpret_cast<uint16_t*>(zeros));
    else
      hipLaunchKernelGGL(q6_k_repack_kernel, dim3(grid), dim3(256), 0, s, reinterpret_cast<const uint16_t*>(blocks),
                         total, reinterpret_cast<uint8_t*>(codes), reinterpret_cast<uint16_t*>(scales));
    return hipGetLastError();
  }
  switch (type) {
    case kQ4_0: return launch_repack<kQ4_0>(blocks, N, K, codes, scales, zeros, s);
    case kQ4_1: return launch_repack<kQ4_1>(blocks, N, K, codes, scales, zeros, s);
    case kQ8_0: return launch_repack<kQ8_0>(blocks, N, K, codes, scales, zeros, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace rlx
