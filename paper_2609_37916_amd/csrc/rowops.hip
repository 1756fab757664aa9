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
// Every row kernel gives one wave to one row; lane l owns columns l, l+64, ...
// so each wave-wide access is one contiguous run of the row.  LayerNorm
// statistics are fp32, two passes over registers (mean, then centred sum of
// squares), with butterfly wave reductions.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace rlx {
namespace {

constexpr int kMaxCols = 16;  // H <= 1024

__global__ __launch_bounds__(1024) void mask_scan_kernel(const uint8_t* mask, int B, int S, int* cu, int* tok_src,
                                                         int* tok_dst) {
  extern __shared__ int offs[];  // [B+1]
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
  if (threadIdx.x == 0) {
    int run = 0;
    for (int b = 0; b < B; ++b) {
      const int c = offs[b];
      offs[b] = run;
      run += c;
    }
    offs[B] = run;
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

template <typename T>
__device__ __forceinline__ void ln_store(float (&v)[kMaxCols], int ncol, const float* gamma, const float* beta,
                                         float eps, int H, T* out) {
  const int lane = threadIdx.x & 63;
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxCols; ++i)
    if (i < ncol) sum += v[i];
  const float mean = wave_sum(sum) / (float)H;
  float sq = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxCols; ++i)
    if (i < ncol) {
      const float c = v[i] - mean;
      sq += c * c;
    }
  const float var = wave_sum(sq) / (float)H;
  const float rstd = 1.0f / sqrtf(var + eps);
#pragma unroll
  for (int i = 0; i < kMaxCols; ++i)
    if (i < ncol) {
      const int c = i * 64 + lane;
      ElemTraits<T>::store(out + c, (v[i] - mean) * rstd * gamma[c] + beta[c]);
    }
}

template <typename T>
__global__ __launch_bounds__(256) void embed_ln_kernel(const int* ids, const T* word, const T* pos, const T* type,
                                                       const float* gamma, const float* beta, float eps, int vocab,
                                                       int S, int H, const int* tok_src, const int* n_dev, int n_max,
                                                       T* x) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n = min(n_max, *n_dev);
  if (t >= n) return;
  const int lane = threadIdx.x & 63;
  const int src = tok_src[t];
  const int s = src % S;
  const int id = min(max(ids[src], 0), vocab - 1);
  const int ncol = H >> 6;
  float v[kMaxCols];
#pragma unroll
  for (int i = 0; i < kMaxCols; ++i)
    if (i < ncol) {
      const int c = i * 64 + lane;
      v[i] = ElemTraits<T>::load(word + (size_t)id * H + c) + ElemTraits<T>::load(pos + (size_t)s * H + c) +
             ElemTraits<T>::load(type + c);
    }
  ln_store<T>(v, ncol, gamma, beta, eps, H, x + (size_t)t * H);
}

template <typename T>
__global__ __launch_bounds__(256) void layer_norm_kernel(const T* a, const float* gamma, const float* beta, float eps,
                                                         int H, const int* n_dev, int n_max, T* y) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n = n_dev ? min(n_max, *n_dev) : n_max;
  if (t >= n) return;
  const int lane = threadIdx.x & 63;
  const int ncol = H >> 6;
  float v[kMaxCols];
#pragma unroll
  for (int i = 0; i < kMaxCols; ++i)
    if (i < ncol) v[i] = ElemTraits<T>::load(a + (size_t)t * H + i * 64 + lane);
  ln_store<T>(v, ncol, gamma, beta, eps, H, y + (size_t)t * H);
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

// One block of 256 threads per sequence: two row groups of 128 threads sum
// alternate rows, then the block forms the mean and its L2 norm.
template <typename T>
__global__ __launch_bounds__(256) void pool_l2_kernel(const T* x, int H, const int* cu, float* out) {
  __shared__ float part[1024];
  __shared__ float red[4];
  const int b = blockIdx.x;
  const int r0 = cu[b], L = cu[b + 1] - r0;
  const int g = threadIdx.x >> 7, c0 = threadIdx.x & 127;
  float acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = 0.0f;
  for (int r = g; r < L; r += 2) {
    const T* row = x + (size_t)(r0 + r) * H;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = c0 + 128 * j;
      if (c < H) acc[j] += ElemTraits<T>::load(row + c);
    }
  }
  if (g == 1) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = c0 + 128 * j;
      if (c < H) part[c] = acc[j];
    }
  }
  __syncthreads();
  const float denom = fmaxf((float)L, 1e-9f);
  float ss = 0.0f;
  if (g == 0) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = c0 + 128 * j;
      if (c < H) {
        acc[j] = (acc[j] + part[c]) / denom;
        ss += acc[j] * acc[j];
      }
    }
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float inv = 1.0f / fmaxf(sqrtf(tot), 1e-12f);
  if (g == 0) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = c0 + 128 * j;
      if (c < H) out[(size_t)b * H + c] = acc[j] * inv;
    }
  }
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

hipError_t launch_mask_scan(const uint8_t* mask, int B, int S, int* cu, int* tok_src, int* tok_dst, hipStream_t s) {
  hipLaunchKernelGGL(mask_scan_kernel, dim3(1), dim3(1024), (size_t)(B + 1) * sizeof(int), s, mask, B, S, cu,
                     tok_src, tok_dst);
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

hipError_t launch_pool_l2(const void* x, int H, const int* cu, int B, float* out, DType dt, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if (dt == DType::BF16)
    hipLaunchKernelGGL(pool_l2_kernel<bf16_t>, dim3(B), dim3(256), 0, s, (const bf16_t*)x, H, cu, out);
  else
    hipLaunchKernelGGL(pool_l2_kernel<float>, dim3(B), dim3(256), 0, s, (const float*)x, H, cu, out);
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
