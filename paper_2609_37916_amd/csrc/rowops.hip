// Row-wise, HBM-bound kernels of the encoder forward: mask scan and token
// compaction, embedding gather + LayerNorm, LayerNorm, masked mean-pool + L2
// normalisation, and the hidden-state scatter.
//
// Token compaction: attention excludes masked keys, so masked tokens never
// influence a real token; every row-local step (projections, LayerNorm, FFN)
// can therefore run on the real tokens only.  The mask scan lists them once
// per forward (tok_src, prefix offsets cu), all later kernels work on that
// dense list, and pooling / the hidden-state output map back.
//
// Every row kernel gives one wave to one row; lane l owns the 16-byte chunks
// l, l+64, ... of the row, so each wave-wide access is one contiguous run.  LayerNorm
// statistics are fp32, two passes over registers (mean, then centred sum of
// squares), with butterfly wave reductions.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace rlx {
namespace {

__global__ __launch_bounds__(1024) void mask_scan_kernel(const uint8_t* mask, int B, int S, int* cu, int* tok_src,
                                                         int* tok_dst, int* order) {
  extern __shared__ int offs[];  // [B+1]: token counts, then their exclusive prefix; then [B] ranks
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const uint64_t below = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
  for (int b = wave; b < B; b += nw) {
    int cnt = 0;
    for (int s0 = 0; s0 < S; s0 += 64) {
      const int s = s0 + lane;
      const bool v = s < S && mask[(size_t)b * S + s] != 0;
      cnt += __popcll(__ballot(v));
    }
    if (lane == 0) offs[b] = cnt;
  }
  __syncthreads();
  // Sequences by token count, longest first (ties by index), for kernels that
  // give each sequence its own blocks: launched in this order, the long ones
  // are placed first and get a CU each.  Small batches only (quadratic).
  if (order) {
    // thread (t, part): sequences u = part, part + P, ... of the comparison
    // for sequence t; the P = blockDim/B partial ranks are summed in LDS
    const int P = max(1, (int)blockDim.x / B);
    int* rank = offs + B + 1;  // [B]
    for (int t = threadIdx.x; t < B; t += blockDim.x) rank[t] = 0;
    __syncthreads();
    const int t = threadIdx.x / P, part = threadIdx.x % P;
    if (t < B) {
      const int c = offs[t];
      int r = 0;
#pragma unroll 4
      for (int u = part; u < B; u += P) r += (offs[u] > c || (offs[u] == c && u < t)) ? 1 : 0;
      atomicAdd(&rank[t], r);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < B; i += blockDim.x) order[rank[i]] = i;
    __syncthreads();
  }
  // exclusive prefix of the counts: wave 0, 64 sequences at a time
  if (wave == 0) {
    int carry = 0;
    for (int c0 = 0; c0 < B; c0 += 64) {
      const int v = c0 + lane < B ? offs[c0 + lane] : 0;
      int incl = v;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int n = __shfl_up(incl, o, 64);
        if (lane >= o) incl += n;
      }
      if (c0 + lane < B) offs[c0 + lane] = carry + incl - v;
      carry += __shfl(incl, 63, 64);
    }
    if (lane == 0) offs[B] = carry;
  }
  __syncthreads();
  for (int i = threadIdx.x; i <= B; i += blockDim.x) cu[i] = offs[i];
  for (int b = wave; b < B; b += nw) {
    int base = offs[b];
    for (int s0 = 0; s0 < S; s0 += 64) {
      const int s = s0 + lane;
      const bool v = s < S && mask[(size_t)b * S + s] != 0;
      const uint64_t bal = __ballot(v);
      const int rank = __popcll(bal & below);
      if (s < S) {
        const int src = b * S + s;
        if (v) tok_src[base + rank] = src;
        tok_dst[src] = v ? base + rank : -1;
      }
      base += __popcll(bal);
    }
  }
}

// Row held by one wave as 16-byte chunks: lane owns chunks lane, lane+64, ...
// (EPC elements each), so every wave-wide load or store is one contiguous run.
template <typename T> struct Chunk;
template <> struct Chunk<bf16_t> {
  static constexpr int EPC = 8;
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
template <> struct Chunk<float> {
  static constexpr int EPC = 4;
  static __device__ __forceinline__ void load(const float* p, float v[4]) {
    const float4 u = *reinterpret_cast<const float4*>(p);
    v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
  }
  static __device__ __forceinline__ void store(float* p, const float v[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
};

// Chunks per lane: H <= 1024 gives at most 2 (bf16) or 4 (f32).
template <typename T> constexpr int kMaxCpl = 8 / Chunk<T>::EPC * 2;

// LayerNorm of the wave's row held in v (fp32), written as T.
template <typename T>
__device__ __forceinline__ void ln_row_store(float (&v)[kMaxCpl<T>][Chunk<T>::EPC], int H, const float* gamma,
                                             const float* beta, float eps, T* out) {
  constexpr int EPC = Chunk<T>::EPC, CPL = kMaxCpl<T>;
  const int lane = threadIdx.x & 63;
  const int nch = H / EPC;
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < CPL; ++i)
    if (lane + 64 * i < nch)
#pragma unroll
      for (int e = 0; e < EPC; ++e) sum += v[i][e];
  const float mean = wave_sum(sum) / (float)H;
  float sq = 0.0f;
#pragma unroll
  for (int i = 0; i < CPL; ++i)
    if (lane + 64 * i < nch)
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        const float c = v[i][e] - mean;
        sq += c * c;
      }
  const float rstd = 1.0f / sqrtf(wave_sum(sq) / (float)H + eps);
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int ch = lane + 64 * i;
    if (ch < nch) {
      float o[EPC];
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        const int c = ch * EPC + e;
        o[e] = (v[i][e] - mean) * rstd * gamma[c] + beta[c];
      }
      Chunk<T>::store(out + ch * EPC, o);
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void embed_ln_kernel(const int* ids, const T* word, const T* pos, const T* type,
                                                       const float* gamma, const float* beta, float eps, int vocab,
                                                       int S, int H, const int* tok_src, const int* n_dev, int n_max,
                                                       T* x) {
  constexpr int EPC = Chunk<T>::EPC, CPL = kMaxCpl<T>;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n = min(n_max, *n_dev);
  if (t >= n) return;
  const int lane = threadIdx.x & 63;
  const int src = tok_src[t];
  const int s = src % S;
  const int id = min(max(ids[src], 0), vocab - 1);
  const int nch = H / EPC;
  float v[CPL][EPC];
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int ch = lane + 64 * i;
    if (ch < nch) {
      float a[EPC], b[EPC], c[EPC];
      Chunk<T>::load(word + (size_t)id * H + ch * EPC, a);
      Chunk<T>::load(pos + (size_t)s * H + ch * EPC, b);
      Chunk<T>::load(type + ch * EPC, c);
#pragma unroll
      for (int e = 0; e < EPC; ++e) v[i][e] = a[e] + b[e] + c[e];
    }
  }
  ln_row_store<T>(v, H, gamma, beta, eps, x + (size_t)t * H);
}

template <typename T>
__global__ __launch_bounds__(256) void layer_norm_kernel(const T* a, const float* gamma, const float* beta, float eps,
                                                         int H, const int* n_dev, int n_max, T* y) {
  constexpr int EPC = Chunk<T>::EPC, CPL = kMaxCpl<T>;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n = n_dev ? min(n_max, *n_dev) : n_max;
  if (t >= n) return;
  const int lane = threadIdx.x & 63;
  const int nch = H / EPC;
  float v[CPL][EPC];
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int ch = lane + 64 * i;
    if (ch < nch) Chunk<T>::load(a + (size_t)t * H + ch * EPC, v[i]);
  }
  ln_row_store<T>(v, H, gamma, beta, eps, y + (size_t)t * H);
}

template <typename T>
__global__ __launch_bounds__(256) void gather_rows_kernel(const T* hidden, int H, const int* tok_src, const int* n_dev,
                                                          int n_max, T* x) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n = min(n_max, *n_dev);
  if (t >= n) return;
  const int lane = threadIdx.x & 63;
  const T* src = hidden + (size_t)tok_src[t] * H;
  for (int c = lane; c < H; c += 64) x[(size_t)t * H + c] = src[c];
}

// Masked mean-pool + L2 normalisation: one block of 1024 threads (16 waves)
// per sequence; wave w sums rows w, w+16, ... with 16-byte chunk loads, the
// 16 partial rows are combined in LDS, then the block forms the mean and its
// norm.
constexpr int kMaxPoolRows = 512;  // the longest sequence
// With x_stats the rows are pre-LayerNorm values with their partial
// statistics (deferred LayerNorm): the block averages (x - mean) * rstd and
// applies gamma and beta to the average.
template <typename T>
__global__ __launch_bounds__(1024) void pool_l2_kernel(const T* x, int H, const int* cu, float* out,
                                                       const float2* x_stats, const float* gamma, const float* beta,
                                                       float eps) {
  constexpr int EPC = Chunk<T>::EPC, CPL = kMaxCpl<T>;
  extern __shared__ float part[];  // [16][H]
  __shared__ float red[16];
  __shared__ float2 row_st[kMaxPoolRows];  // (mean, rstd) per row of a deferred-LayerNorm input
  const int b = blockIdx.x;
  const int r0 = cu[b], L = cu[b + 1] - r0;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (x_stats) {  // all rows' statistics in one round of loads, one row per thread
    for (int r = threadIdx.x; r < L; r += 1024) row_st[r] = row_ln_stats(x_stats + (size_t)(r0 + r) * (H >> 6), H >> 6, eps);
    __syncthreads();
  }
  const int nch = H / EPC;
  float acc[CPL][EPC];
#pragma unroll
  for (int i = 0; i < CPL; ++i)
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[i][e] = 0.0f;
  for (int r = wave; r < L; r += 16) {
    const T* row = x + (size_t)(r0 + r) * H;
    // (0, 1) leaves plain rows as they are
    const float2 st = x_stats ? row_st[r] : make_float2(0.0f, 1.0f);
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int ch = lane + 64 * i;
      if (ch < nch) {
        float v[EPC];
        Chunk<T>::load(row + ch * EPC, v);
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[i][e] += (v[e] - st.x) * st.y;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int ch = lane + 64 * i;
    if (ch < nch)
#pragma unroll
      for (int e = 0; e < EPC; ++e) part[wave * H + ch * EPC + e] = acc[i][e];
  }
  __syncthreads();
  const float denom = fmaxf((float)L, 1e-9f);
  const int c = threadIdx.x;
  float mean = 0.0f;
  if (c < H) {
    float sum = 0.0f;
#pragma unroll
    for (int w = 0; w < 16; ++w) sum += part[w * H + c];
    mean = sum / denom;
    if (x_stats) mean = L > 0 ? fmaf(gamma[c], mean, beta[c]) : 0.0f;
  }
  const float ss = wave_sum(mean * mean);
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  float tot = 0.0f;
#pragma unroll
  for (int w = 0; w < 16; ++w) tot += red[w];
  const float inv = 1.0f / fmaxf(sqrtf(tot), 1e-12f);
  if (c < H) out[(size_t)b * H + c] = mean * inv;
}

template <typename T>
__global__ __launch_bounds__(256) void scatter_hidden_kernel(const T* x, int H, const int* tok_dst, int n_tok,
                                                             float* out) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= n_tok) return;
  const int lane = threadIdx.x & 63;
  const int t = tok_dst[i];
  for (int c = lane; c < H; c += 64)
    out[(size_t)i * H + c] = t >= 0 ? ElemTraits<T>::load(x + (size_t)t * H + c) : 0.0f;
}

inline int blocks_for_rows(int rows) { return (rows + 3) / 4; }

}  // namespace

hipError_t launch_mask_scan(const uint8_t* mask, int B, int S, int* cu, int* tok_src, int* tok_dst, int* order,
                            hipStream_t s) {
  hipLaunchKernelGGL(mask_scan_kernel, dim3(1), dim3(1024), (size_t)(2 * B + 1) * sizeof(int), s, mask, B, S, cu,
                     tok_src, tok_dst, B <= kMaxOrderedBatch ? order : nullptr);
  return hipGetLastError();
}

hipError_t launch_embed_ln(const int* ids, const void* word, const void* pos, const void* type, const float* gamma,
                           const float* beta, float eps, int vocab, int S, int H, const int* tok_src,
                           const int* n_dev, int n_max, void* x, DType dt, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dt == DType::BF16)
    hipLaunchKernelGGL(embed_ln_kernel<bf16_t>, dim3(blocks_for_rows(n_max)), dim3(256), 0, s, ids,
                       (const bf16_t*)word, (const bf16_t*)pos, (const bf16_t*)type, gamma, beta, eps, vocab, S, H,
                       tok_src, n_dev, n_max, (bf16_t*)x);
  else
    hipLaunchKernelGGL(embed_ln_kernel<float>, dim3(blocks_for_rows(n_max)), dim3(256), 0, s, ids, (const float*)word,
                       (const float*)pos, (const float*)type, gamma, beta, eps, vocab, S, H, tok_src, n_dev, n_max,
                       (float*)x);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const void* hidden, int H, const int* tok_src, const int* n_dev, int n_max, void* x,
                              DType dt, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dt == DType::BF16)
    hipLaunchKernelGGL(gather_rows_kernel<bf16_t>, dim3(blocks_for_rows(n_max)), dim3(256), 0, s,
                       (const bf16_t*)hidden, H, tok_src, n_dev, n_max, (bf16_t*)x);
  else
    hipLaunchKernelGGL(gather_rows_kernel<float>, dim3(blocks_for_rows(n_max)), dim3(256), 0, s, (const float*)hidden,
                       H, tok_src, n_dev, n_max, (float*)x);
  return hipGetLastError();
}

hipError_t launch_layer_norm(const void* a, const float* gamma, const float* beta, float eps, int H,
                             const int* n_dev, int n_max, void* y, DType dt, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dt == DType::BF16)
    hipLaunchKernelGGL(layer_norm_kernel<bf16_t>, dim3(blocks_for_rows(n_max)), dim3(256), 0, s, (const bf16_t*)a,
                       gamma, beta, eps, H, n_dev, n_max, (bf16_t*)y);
  else
    hipLaunchKernelGGL(layer_norm_kernel<float>, dim3(blocks_for_rows(n_max)), dim3(256), 0, s, (const float*)a, gamma,
                       beta, eps, H, n_dev, n_max, (float*)y);
  return hipGetLastError();
}

hipError_t launch_pool_l2(const void* x, int H, const int* cu, int B, float* out, DType dt, hipStream_t s,
                          const float2* x_stats, const float* gamma, const float* beta, float eps) {
  if (B <= 0) return hipSuccess;
  const size_t lds = (size_t)16 * H * sizeof(float);
  if (dt == DType::BF16)
    hipLaunchKernelGGL(pool_l2_kernel<bf16_t>, dim3(B), dim3(1024), lds, s, (const bf16_t*)x, H, cu, out, x_stats,
                       gamma, beta, eps);
  else if (x_stats)
    return hipErrorInvalidValue;
  else
    hipLaunchKernelGGL(pool_l2_kernel<float>, dim3(B), dim3(1024), lds, s, (const float*)x, H, cu, out, nullptr,
                       nullptr, nullptr, 0.0f);
  return hipGetLastError();
}

hipError_t launch_scatter_hidden(const void* x, int H, const int* tok_dst, int n_tok, float* out, DType dt,
                                 hipStream_t s) {
  if (n_tok <= 0) return hipSuccess;
  if (dt == DType::BF16)
    hipLaunchKernelGGL(scatter_hidden_kernel<bf16_t>, dim3(blocks_for_rows(n_tok)), dim3(256), 0, s,
                       (const bf16_t*)x, H, tok_dst, n_tok, out);
  else
    hipLaunchKernelGGL(scatter_hidden_kernel<float>, dim3(blocks_for_rows(n_tok)), dim3(256), 0, s, (const float*)x, H,
                       tok_dst, n_tok, out);
  return hipGetLastError();
}

}  // namespace rlx
