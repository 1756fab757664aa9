// Device helpers shared by the gfx950 kernels: bf16 storage conversions,
// MFMA operand types, wave reductions.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rlx {

// Launch log (RLX_LOG=1 in the environment, read again at every C-ABI entry
// point): each launch prints its kernel with the parameters that chose it,
// its grid, block and dynamic LDS, to stderr.  Launches recorded into a HIP
// graph print once, when recorded.
extern bool g_log_launches;
void log_launch(const char* kernel, dim3 grid, dim3 block, size_t lds, const char* fmt, ...)
    __attribute__((format(printf, 5, 6)));
#define RLX_LOG_LAUNCH(kernel, grid, block, lds, ...)                      \
  do {                                                                     \
    if (::rlx::g_log_launches) ::rlx::log_launch(kernel, grid, block, lds, __VA_ARGS__); \
  } while (0)

typedef uint16_t bf16_t;  // bfloat16 storage (upper half of an IEEE binary32)

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Round to nearest, ties to even; NaN stays NaN.  gfx950 converts in hardware
// (v_cvt_pk_bf16_f32, two values per instruction); a bit-twiddling version
// with a NaN test compiles to a divergent branch per element.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ float f16_bits_to_f32(uint16_t h) {
  _Float16 v;
  __builtin_memcpy(&v, &h, 2);
  return (float)v;
}

template <typename T> struct ElemTraits;
template <> struct ElemTraits<float> {
  static __device__ __forceinline__ float load(const float* p) { return *p; }
  static __device__ __forceinline__ void store(float* p, float v) { *p = v; }
};
template <> struct ElemTraits<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t* p) { return bf16_to_f32(*p); }
  static __device__ __forceinline__ void store(bf16_t* p, float v) { *p = f32_to_bf16(v); }
};

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// erf by Abramowitz & Stegun, Handbook of Mathematical Functions, formula
// 7.1.28 (Hastings): for t >= 0, erf(t) = 1 - (1 + a1 t + ... + a6 t^6)^-16
// with |error| <= 3e-7.  Six FMAs, four squarings and one reciprocal -- about a
// third of the instructions of the library erff, which matters because the
// FFN-up epilogue evaluates it once per output element.
__device__ __forceinline__ float erf_as7128(float t) {
  const float a = fabsf(t);
  float p = 0.0000430638f;
  p = fmaf(p, a, 0.0002765672f);
  p = fmaf(p, a, 0.0001520143f);
  p = fmaf(p, a, 0.0092705272f);
  p = fmaf(p, a, 0.0422820123f);
  p = fmaf(p, a, 0.0705230784f);
  p = fmaf(p, a, 1.0f);
  p = p * p;  // ^2
  p = p * p;  // ^4
  p = p * p;  // ^8
  p = p * p;  // ^16 (overflow to +inf gives erf = 1, the correct limit)
  const float e = 1.0f - __builtin_amdgcn_rcpf(p);
  return copysignf(e, t);
}

// GELU(x) = x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2))
__device__ __forceinline__ float gelu_erf(float x) {
  const float h = 0.5f * x;
  return fmaf(h, erf_as7128(x * 0.70710678118654752f), h);
}

// Deferred LayerNorm (Section VIII-B's post-LN blocks, computed by the
// consumers of an activation): a row of `np` * 64 columns carries, per 64
// columns j, (mean_j, sum over those columns of (a - mean_j)^2).  They merge
// into the row's mean and 1/sqrt(var + eps) with the pairwise update of Chan,
// Golub and LeVeque (equal counts): mean = average of mean_j,
// M2 = sum_j M2_j + 64 * sum_j (mean_j - mean)^2, var = M2 / (64 np).
constexpr int kLnMaxParts = 16;  // rows of up to 1024 columns
__device__ __forceinline__ void load_ln_parts(const float2* part, int np, float2 (&v)[kLnMaxParts]) {
#pragma unroll
  for (int j = 0; j < kLnMaxParts; ++j) v[j] = j < np ? part[j] : make_float2(0.0f, 0.0f);
}
__device__ __forceinline__ float2 merge_ln_parts(const float2 (&v)[kLnMaxParts], int np, float eps) {
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < kLnMaxParts; ++j) s += v[j].x;
  const float mean = s / (float)np;
  float m2 = 0.0f;
#pragma unroll
  for (int j = 0; j < kLnMaxParts; ++j)
    if (j < np) {
      const float d = v[j].x - mean;
      m2 += fmaf(64.0f * d, d, v[j].y);
    }
  return make_float2(mean, 1.0f / sqrtf(m2 / (float)(64 * np) + eps));
}
__device__ __forceinline__ float2 row_ln_stats(const float2* part, int np, float eps) {
  float2 v[kLnMaxParts];
  load_ln_parts(part, np, v);
  return merge_ln_parts(v, np, eps);
}
// The same from statistics staged in LDS, for np parts known at compile
// time (np even: rows of an even number of 64-column parts): the np / 2
// 16-byte pairs are read at once (one LDS round trip), the sums are taken as
// trees rather than one serial chain, and the reciprocal square root is the
// hardware one (its argument is at least eps, never denormal).
template <int NP>
__device__ __forceinline__ float2 merge_ln_lds_n(const float2* part, float eps) {
  static_assert(NP % 2 == 0 && NP >= 2 && NP <= kLnMaxParts, "even part count");
  constexpr int NQ = NP / 2;
  const float4* q = reinterpret_cast<const float4*>(part);
  float4 v[NQ];
#pragma unroll
  for (int j = 0; j < NQ; ++j) v[j] = q[j];
  float a[NQ];
#pragma unroll
  for (int j = 0; j < NQ; ++j) a[j] = v[j].x + v[j].z;
#pragma unroll
  for (int w = 1; w < NQ; w *= 2)
#pragma unroll
    for (int j = 0; j + w < NQ; j += 2 * w) a[j] += a[j + w];
  const float mean = a[0] * (1.0f / NP);
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    const float d0 = v[j].x - mean, d1 = v[j].z - mean;
    a[j] = fmaf(64.0f * d0, d0, fmaf(64.0f * d1, d1, v[j].y + v[j].w));
  }
#pragma unroll
  for (int w = 1; w < NQ; w *= 2)
#pragma unroll
    for (int j = 0; j + w < NQ; j += 2 * w) a[j] += a[j + w];
  return make_float2(mean, __builtin_amdgcn_rsqf(fmaf(a[0], 1.0f / (64.0f * NP), eps)));
}
// Any part count: all kLnMaxParts entries are read at once (16-byte aligned,
// 128 readable bytes: the caller pads) and the ones past np are masked.
__device__ __forceinline__ float2 merge_ln_lds_any(const float2* part, int np, float eps) {
  const float4* q = reinterpret_cast<const float4*>(part);
  float4 v[kLnMaxParts / 2];
#pragma unroll
  for (int j = 0; j < kLnMaxParts / 2; ++j) v[j] = q[j];
  const float inv_np = __builtin_amdgcn_rcpf((float)np);
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < kLnMaxParts / 2; ++j) s += 2 * j < np ? v[j].x + v[j].z : 0.0f;
  const float mean = s * inv_np;
  float m2 = 0.0f;
#pragma unroll
  for (int j = 0; j < kLnMaxParts / 2; ++j) {
    const float d0 = v[j].x - mean, d1 = v[j].z - mean;
    const float t = fmaf(64.0f * d0, d0, fmaf(64.0f * d1, d1, v[j].y + v[j].w));
    m2 += 2 * j < np ? t : 0.0f;
  }
  return make_float2(mean, rsqrtf(fmaf(m2, inv_np * (1.0f / 64.0f), eps)));
}
// np is the same across the wave, so the switch is a scalar branch.
__device__ __forceinline__ float2 merge_ln_lds(const float2* part, int np, float eps) {
  switch (np) {
    case 2: return merge_ln_lds_n<2>(part, eps);
    case 4: return merge_ln_lds_n<4>(part, eps);
    case 6: return merge_ln_lds_n<6>(part, eps);
    case 8: return merge_ln_lds_n<8>(part, eps);
    case 12: return merge_ln_lds_n<12>(part, eps);
    case 16: return merge_ln_lds_n<16>(part, eps);
    default: return merge_ln_lds_any(part, np, eps);
  }
}

// Sum over each group of 8 consecutive lanes, by DPP lane swaps (no LDS):
// quad_perm [1,0,3,2] (xor 1), quad_perm [2,3,0,1] (xor 2), then the half-row
// mirror (lane i <-> 7-i of each 8), which pairs the two quads' sums.
__device__ __forceinline__ float dpp_sum8(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x141, 0xF, 0xF, false));
  return v;
}

// ---------------------------------------------------------------------------
// Direct-to-LDS loads and explicit waits
// ---------------------------------------------------------------------------
// global_load_lds: each lane's 16 (or 4) bytes go from global memory straight
// into LDS at m0 + lane * 16 (* 4).  Inline assembly keeps the compiler from
// inserting a full vmcnt wait before every later LDS read (it cannot tell
// which LDS bytes the load writes); the kernels place their own waits.  M0 is
// used by nothing else in these kernels.
__device__ __forceinline__ void lds_dma16(const void* g, uint32_t lds_addr) {
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds_addr)
               : "memory", "m0");
#pragma clang diagnostic pop
}
__device__ __forceinline__ void lds_dma4(const void* g, uint32_t lds_addr) {
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off" ::"v"(g), "s"(lds_addr)
               : "memory", "m0");
#pragma clang diagnostic pop
}

// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Wait until this wave's LDS reads (and scalar loads) have returned.
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14)); }

// ahead (<= MAXA) later stages of LPS loads each may stay in flight
template <int LPS, int MAXA>
__device__ __forceinline__ void wait_stage(int ahead) {
  if constexpr (MAXA > 0) {
    if (ahead >= MAXA) {
      wait_vmcnt<MAXA * LPS>();
      return;
    }
    wait_stage<LPS, MAXA - 1>(ahead);
  } else {
    wait_vmcnt<0>();
  }
}

// wait_stage, with `extra` (0 .. 7) younger loads issued after the later
// stages also allowed to stay in flight (more: waits for everything).
template <int LPS, int MAXA, int E>
__device__ __forceinline__ void wait_stage_e(int ahead) {
  if constexpr (MAXA > 0) {
    if (ahead >= MAXA) {
      wait_vmcnt<MAXA * LPS + E>();
      return;
    }
    wait_stage_e<LPS, MAXA - 1, E>(ahead);
  } else {
    wait_vmcnt<E>();
  }
}
template <int LPS, int MAXA>
__device__ __forceinline__ void wait_stage_plus(int ahead, int extra) {
  switch (extra) {
    case 0: wait_stage_e<LPS, MAXA, 0>(ahead); break;
    case 1: wait_stage_e<LPS, MAXA, 1>(ahead); break;
    case 2: wait_stage_e<LPS, MAXA, 2>(ahead); break;
    case 3: wait_stage_e<LPS, MAXA, 3>(ahead); break;
    case 4: wait_stage_e<LPS, MAXA, 4>(ahead); break;
    case 5: wait_stage_e<LPS, MAXA, 5>(ahead); break;
    case 6: wait_stage_e<LPS, MAXA, 6>(ahead); break;
    case 7: wait_stage_e<LPS, MAXA, 7>(ahead); break;
    default: wait_vmcnt<0>(); break;
  }
}

// LDS byte address of a __shared__ pointer (for m0).
__device__ __forceinline__ uint32_t lds_addr_of(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)p;
}

// Reinterpret 16 bytes as eight bf16 MFMA operands.
__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

}  // namespace rlx
