// Internal launch interface between the C ABI (capi.hip) and the kernels.
// Launchers assume their arguments were validated by the caller; they only
// enqueue work and return the launch status.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace rlx {

enum class DType : int { F32 = 0, BF16 = 1 };
// Weight layouts of the dequantising matmul: Int8 per-channel scales; Int4
// group-32 scale and zero-point, W = (q - z) s; Int8G int8 codes with group-32
// scales, W = q s; Int4M group-32 scale and min, W = q s + m; Int8G16 int8
// codes with group-16 scales, W = q s.
enum class Quant : int { None = 0, Int8 = 1, Int4 = 2, Int8G = 3, Int4M = 4, Int8G16 = 5 };
__host__ __device__ constexpr bool quant_int8(Quant q) {
  return q == Quant::Int8 || q == Quant::Int8G || q == Quant::Int8G16;
}
// Weights per scale of a grouped layout.
__host__ __device__ constexpr int quant_group_size(Quant q) { return q == Quant::Int8G16 ? 16 : 32; }
__host__ __device__ constexpr bool quant_int4(Quant q) { return q == Quant::Int4 || q == Quant::Int4M; }
enum class Epi : int { None = 0, Bias = 1, BiasGelu = 2, BiasResidual = 3 };

struct GemmParams {
  const void* x;         // [M,K] activations (dtype)
  const void* w;         // weights in the layout of `quant`
  const void* scales;    // f16 (int8: [N]; int4: [N,K/32])
  const void* zeros;     // f16 [N,K/32] (int4)
  const float* bias;     // f32 [N]
  const void* residual;  // [M,N] (dtype, or f32 with y_f32)
  void* y;               // [M,N] (dtype, or f32 with y_f32)
  int M, N, K;           // M is an upper bound when m_dev is set
  const int* m_dev;      // optional device-side row count (rows >= *m_dev are skipped)
  DType dtype;
  Quant quant;
  Epi epi;
  int tile;              // 0: choose automatically; otherwise a GemmTile value (tuning)
  int x_head_rows;       // 0: x is row-major [M,K]; > 0: x is head-major [K/32][x_head_rows][32]
                         // (dense bf16 only), as written by the fused attention
  // Deferred LayerNorm (bf16 activations).  A post-LN activation can travel
  // as its pre-norm rows a plus, per row and per 64 columns, the mean and the
  // centred sum of squares of the stored values (float2 [rows][cols/64],
  // "partial statistics"); whoever reads it applies the norm.  Dense weights
  // take gamma folded into W; quantised weights cannot, so their activation
  // travels gamma-scaled (gamma[k] * a[k]) instead.
  //  x_stats: x is such an activation and the product carries gamma (in W or in x):
  //           y = rstd[m] * (acc - mean[m] * fold_u[n]) + bias[n], then the epilogue,
  //           fold_u[n] = sum_k gamma_k W_nk
  //  res_stats: the residual is such an activation:
  //           residual[m,n] = (a[m,n] - mean[m]) * rstd[m] * res_gamma[n] + res_beta[n]
  //           (res_scaled: stored as gamma * a, so rstd[m] * (r - mean[m] * res_gamma[n]) + res_beta[n])
  //  y_stats: also write the partial statistics of the stored y
  //           (y_gamma: store y_gamma[n] * y; the statistics stay those of y)
  const float2* x_stats;
  const float* fold_u;
  const float2* res_stats;
  const float* res_gamma;
  const float* res_beta;
  float2* y_stats;
  const float* y_gamma;
  bool res_scaled;
  float ln_eps;
  bool y_f32;            // bf16 x with an f32 output (and residual); not with the deferred-LayerNorm fields
};
// Names for the launch log.
inline const char* epi_name(Epi e) {
  return e == Epi::None ? "none" : e == Epi::Bias ? "bias" : e == Epi::BiasGelu ? "bias+gelu" : "bias+residual";
}
inline const char* quant_name(Quant q) {
  return q == Quant::None ? "dense" : q == Quant::Int8 ? "int8" : q == Quant::Int4 ? "int4-zp"
         : q == Quant::Int8G ? "int8-group" : q == Quant::Int8G16 ? "int8-group16" : "int4-min";
}
// True when the deferred-LayerNorm fields are implemented for rows of H columns.
bool gemm_deferred_ln_supported(DType dt, Quant q, int H);
// Deferred LayerNorm with quantised weights, per row n:
//  dense_fold = false (dequantising GEMMs, gamma-scaled inputs): over the
//    effective weights W (the values the matrix cores multiply: q * s for int8
//    per channel, the bf16 rounding of the scheme's dequantisation otherwise)
//    u[n] = sum_k gamma_k W_nk;
//  dense_fold = true (weights dequantised to bf16 with gamma folded in,
//    W'_nk = bf16(gamma_k * d_nk), d the fp32 dequantisation): u[n] = sum_k W'_nk;
//  both: v[n] = bias[n] + sum_k beta_k W_nk.
hipError_t launch_fold_ln_quant(const void* w, Quant q, const void* scales, const void* zeros, int N, int K,
                                const float* gamma, const float* beta, const float* bias, bool dense_fold,
                                float* u_out, float* v_out, hipStream_t s);

// One matrix for launch_dequant_jobs: quantised weights [N,K] (K a multiple
// of 32) to bf16 [N,K] at `out`, each element bf16(gamma[k] * d) when gamma
// is given, else bf16(d), d the fp32 dequantisation (as the GEMM's code
// conversions compute it).
struct DequantJob {
  const void* w; const void* scales; const void* zeros; const float* gamma;
  void* out;
  int N, K;
  Quant quant;
};
// Every job of the device array `jobs` in one launch; max_elems bounds N*K.
hipError_t launch_dequant_jobs(const DequantJob* jobs, int njobs, int max_elems, hipStream_t s);
enum GemmTile : int { kTileAuto = 0, kTile128x128 = 1, kTile64x128 = 2, kTile64x64 = 3, kTile128x64 = 4 };
hipError_t launch_gemm(const GemmParams& p, hipStream_t s);

// Few-row dequantising matmul (gemv.hip): int8 / int4 weights, bf16 x with
// 1 <= M <= 16 rows, N % 16 == 0, K % 128 == 0, M * K * 2 <= 64 KB, 4-byte
// aligned scales and zeros, no device-side row count and no deferred-LayerNorm fields.  launch_gemm takes
// this path by itself whenever it applies.
bool gemv_supported(const GemmParams& p);
hipError_t launch_gemv(const GemmParams& p, hipStream_t s);

// GGUF blocks (type 2 Q4_0, 3 Q4_1, 8 Q8_0) of an [N, K] tensor -> the Int4
// (Q4_0, z = 8), Int4M (Q4_1) or Int8G (Q8_0) layout (gguf.hip).
hipError_t launch_gguf_repack(const void* blocks, int type, int N, int K, void* codes, void* scales, void* zeros,
                              hipStream_t s);

hipError_t launch_dequant_unpack(const void* w, Quant q, const void* scales, const void* zeros, int N, int K,
                                 float* out, hipStream_t s);

struct AttnParams {
  const void* q; const void* k; const void* v; int64_t ld_qkv;
  void* out; int64_t ld_out;
  int B, S, heads;            // S: padded length (max rows per sequence)
  int kind;                   // 0 none, 1 causal, 2 sliding window, 3 custom
  const uint8_t* key_mask;    // [B,S] or null (padded layout only)
  int window;
  float scale;
  const int* cu_seqlens;      // varlen layout: rows of sequence b are [cu[b], cu[b+1]); null = padded layout
  DType dtype;
};
hipError_t launch_attention(const AttnParams& p, hipStream_t s);

// QKV projection fused with attention, one block per (head, sequence), for the
// variable-length layout with at most 128 tokens per sequence, bf16, dense
// weights, head_dim 32:  out[t, h*32+d] = attention of head h over the
// sequence's rows of x * Wqkv^T + bqkv.
struct FusedAttnParams {
  const void* x;        // [T, H] bf16 compact activations
  const void* wqkv;     // [3H, H] bf16
  const float* bqkv;    // [3H]
  const int* cu_seqlens;
  void* out;            // head-major [heads][out_rows][32] bf16
  int out_rows;         // row pitch of one head block (>= real tokens)
  int B, H, heads;
  float scale;
  const int* seq_order;  // optional [B]: the sequences in launch order (longest first)
  // optional [B]: (first row, real tokens) of the sequence at each launch rank,
  // written by the scan that wrote seq_order; read instead of seq_order and
  // cu_seqlens, one dependent load less before a block's first row request
  const int2* rank_rows;
  // optional deferred LayerNorm of x (as GemmParams::x_stats): wqkv holds
  // gamma-scaled weights, bqkv the folded bias, fold_u [3H] the row sums
  const float2* x_stats;
  const float* fold_u;
  float ln_eps;
  // compute units per XCD; set by launch_qkv_attention (0: slots in rank order)
  int cu_per_xcd;
};
hipError_t launch_qkv_attention(const FusedAttnParams& p, hipStream_t s);

// Block-scaled minifloat matmul (ScaledMatMul): y[m,n] = sum_k X(m,k) W(n,k)
// with OCP MX operands (format codes 0 E4M3, 1 E5M2, 2 E2M3, 3 E3M2, 4 E2M1;
// 32 codes per E8M0 scale).  x: [M, K*bits/8], w: [N, K*bits/8] packed rows;
// x_scales [M, K/32], w_scales [N, K/32] (4-byte aligned); y f32 [M, N].
struct MxGemmParams {
  const void* x; const uint8_t* x_scales; int fx;
  const void* w; const uint8_t* w_scales; int fw;
  float* y;
  int M, N, K;
};
bool mx_gemm_supported(int M, int N, int K);  // N, K multiples of 128
hipError_t launch_mx_gemm(const MxGemmParams& p, hipStream_t s);

// Folds a LayerNorm (gamma, beta) into the linear layer that consumes it, for
// the deferred-LayerNorm path: w_out[n,k] = bf16(gamma[k] * w[n,k]),
// u_out[n] = sum_k w_out[n,k], v_out[n] = sum_k beta[k] * w[n,k] + bias[n]
// (sums in fp64).  w: bf16 [N,K].
hipError_t launch_fold_ln_weights(const void* w, int N, int K, const float* gamma, const float* beta,
                                  const float* bias, void* w_out, float* u_out, float* v_out, hipStream_t s);

// Persistent encoder forward (pipe.hip): the whole bf16 forward (embedding,
// `L` post-LN layers with the LayerNorms deferred as in the GEMM kernels,
// pooling) in one launch of resident blocks, each XCD working on its own run
// of sequences.  Shapes it supports: pipe_supported.
constexpr int kPipeHidden = 384;         // hidden size the LDS plan is made for
constexpr int kPipeMaxBatch = 256;
constexpr int kPipeMaxTokens = 32768;    // B * S
constexpr int kPipeMaxRowTiles = kPipeMaxTokens / 64;
constexpr int kPipeMaxLayers = 12;
constexpr int kPipeLdsBytes = 80 * 1024;  // two blocks per CU
// ints of sync words per XCD (a whole number of 4 KB pages)
constexpr int kPipeSyncStride =
    ((64 + kPipeMaxLayers * (kPipeMaxBatch + 3 * kPipeMaxRowTiles)) + 1023) / 1024 * 1024;
struct PipeLayer {
  const bf16_t* wqkv; const float* bqkv; const float* uq;  // layer 0: as given, uq null; later: LN2 folded in
  const bf16_t* wo; const float* bo;
  const float* res_g; const float* res_b;                  // LN2 of the previous layer (the residual); layer 0 null
  const bf16_t* w1; const float* v1; const float* u1;      // LN1 folded in
  const bf16_t* w2; const float* b2;
  const float* ln1_g; const float* ln1_b;
};
struct PipeParams {
  const uint8_t* mask; const int* ids; int B, S;           // mask rows 16-byte aligned, S % 16 == 0
  const bf16_t* word; const bf16_t* pos; const bf16_t* type; const float* emb_g; const float* emb_b; int vocab;
  float eps, scale;
  const PipeLayer* layers; int L;                          // device array
  int H, F, heads;
  bf16_t* X; bf16_t* A; bf16_t* CTX; bf16_t* G; float2* S1; float2* S2; int ctx_rows;
  const float* last_g; const float* last_b;                // LN2 of the last layer
  float* out;                                              // f32 [B, H] pooled
  int* sync;                                               // pipe_sync_bytes(), zero before the first launch
};
struct PipeShape {
  int B, S, H, F, heads, L;
};
bool pipe_supported(const PipeShape& s);
size_t pipe_sync_bytes();
// Clears the sync words, then launches the forward on `grid` blocks.
hipError_t launch_encoder_pipe(const PipeParams& p, int grid, hipStream_t s);
hipError_t init_pipe_attributes();  // raises the kernel's LDS limit (idempotent)

// Raises per-kernel dynamic-LDS limits once per process (idempotent).
hipError_t init_kernel_attributes();

// Mask scan: per-sequence valid counts, offsets and the token compaction maps.
//   cu[0..B]    exclusive prefix of valid counts (cu[B] = valid tokens)
//   tok_src[t]  = b*S + s of compact token t            (t < cu[B])
//   tok_dst[i]  = compact index of padded token i, or -1 (i < B*S)
// order (optional, [B]): the sequences sorted by token count, longest first;
// written only for B <= kMaxOrderedBatch (consumers must then also check B).
// rank_rows (optional, [B], with order): (cu[b], count of b) of b = order[r]
// at entry r, for consumers that walk the sequences in that order.
constexpr int kMaxOrderedBatch = 256;
hipError_t launch_mask_scan(const uint8_t* mask, int B, int S, int* cu, int* tok_src, int* tok_dst, int* order,
                            hipStream_t s, int2* rank_rows = nullptr);

// x[t] = LN(word[id] + pos[s] + type[0]) for compact tokens t < cu[B].
hipError_t launch_embed_ln(const int* ids, const void* word, const void* pos, const void* type, const float* gamma,
                           const float* beta, float eps, int vocab, int S, int H, const int* tok_src,
                           const int* n_dev, int n_max, void* x, DType dt, hipStream_t s);

// The mask scan and the embedding in one kernel (same outputs as both): for
// small masks, where every block can scan the whole mask itself.
constexpr int kEmbedScanMaxMask = 16384;  // B * S
constexpr int kEmbedScanMaxSeq = 512;
inline bool embed_scan_supported(int B, int S) {
  return B <= kMaxOrderedBatch && S <= kEmbedScanMaxSeq && (int64_t)B * S <= kEmbedScanMaxMask;
}
hipError_t launch_embed_scan(const uint8_t* mask, const int* ids, int B, int S, const void* word, const void* pos,
                             const void* type, const float* gamma, const float* beta, float eps, int vocab, int H,
                             int* cu, int* tok_src, int* tok_dst, int* order, void* x, DType dt, hipStream_t s,
                             int2* rank_rows = nullptr);

// x[t] = hidden[tok_src[t]] (row copy) for t < *n_dev.
hipError_t launch_gather_rows(const void* hidden, int H, const int* tok_src, const int* n_dev, int n_max, void* x,
                              DType dt, hipStream_t s);

// y[t] = LN(a[t]) * gamma + beta for t < *n_dev; optional f32 copy of the result.
hipError_t launch_layer_norm(const void* a, const float* gamma, const float* beta, float eps, int H,
                             const int* n_dev, int n_max, void* y, DType dt, hipStream_t s);

// out[b] = normalize(mean over the sequence's compact rows) (f32 [B,H]).
// With x_stats (bf16), x is a deferred-LayerNorm activation (see GemmParams)
// and the rows are normalised with gamma, beta and eps first; gamma_scaled:
// the rows are stored gamma-scaled (quantised-weight encoders).  S bounds the
// sequence lengths (<= 512); with S > 128 each sequence is summed by
// ceil(S / 64) blocks of 64 rows and combined by a second kernel when
// `scratch` holds B * ceil(S / 64) * H floats (scratch_bytes), else by one
// block per sequence.
hipError_t launch_pool_l2(const void* x, int H, const int* cu, int B, float* out, DType dt, hipStream_t s,
                          const float2* x_stats = nullptr, const float* gamma = nullptr,
                          const float* beta = nullptr, float eps = 0.0f, bool gamma_scaled = false, int S = 0,
                          float* scratch = nullptr, size_t scratch_bytes = 0);

// out[b,s,:] = x[tok_dst[b*S+s]] or 0 (f32 [B,S,H]).
hipError_t launch_scatter_hidden(const void* x, int H, const int* tok_dst, int n_tok, float* out, DType dt,
                                 hipStream_t s);

}  // namespace rlx
