/*
 * rlx.h -- C ABI of the MI355X (gfx950) MiniLM-L6-shaped encoder forward.
 *
 * The library computes the forward pass of a BERT-style sentence-embedding
 * encoder (all-MiniLM-L6-v2 shape: hidden 384, 12 heads of 32, FFN 1536,
 * 6 post-LN layers), the workload of the paper's inference evaluation
 * (RLX, arxiv 2609.37916, Section VIII-B), with hand-written HIP kernels.
 *
 * Conventions shared by every entry point
 *  - All tensor pointers are DEVICE pointers unless marked "host".  The
 *    caller owns every buffer it passes; the library never frees or keeps
 *    them beyond the call, except the weights bound by rlx_encoder_create,
 *    which must outlive the encoder handle and keep their values while it
 *    exists (part of them are read once, at create).
 *  - Tensors are dense and row-major unless a row stride is given; strides
 *    are in elements.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Work is enqueued asynchronously on it; results are ready when the
 *    stream is synchronised.
 *  - Every argument is validated before any GPU work is enqueued.  A call
 *    that cannot be executed exactly as asked returns an error and does
 *    nothing: there is no fallback to another algorithm or to the CPU
 *    (the paper's dispatch fails with a diagnostic rather than degrading,
 *    Section IV).  rlx_last_error() then describes the problem.
 *  - bf16 is bfloat16 (upper 16 bits of an IEEE binary32); conversions to
 *    bf16 round to nearest, ties to even.  f16 is IEEE binary16.
 *  - Thread safety: entry points may be called from several host threads;
 *    one encoder handle must not be used by two threads at once.
 */
#ifndef RLX_H_
#define RLX_H_

#include <stddef.h>
#include <stdint.h>

/* The enumerations are int-sized in C and C++ alike.  In C++ they carry the
 * fixed underlying type int32_t, so any int a C caller passes is a value of
 * the enumeration type (an unknown one is rejected by the callee's checks,
 * never undefined behaviour). */
#ifdef __cplusplus
#define RLX_ENUM enum : int32_t
#else
#define RLX_ENUM enum
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef RLX_ENUM {
  RLX_OK = 0,
  RLX_ERR_INVALID_ARG = 1,  /* null pointer, negative size, inconsistent shapes     */
  RLX_ERR_UNSUPPORTED = 2,  /* well-formed request outside what the kernels implement */
  RLX_ERR_HIP = 3,          /* a HIP runtime call or kernel launch failed          */
  RLX_ERR_OOM = 4           /* device allocation failed (encoder workspace)        */
} rlx_status;

typedef RLX_ENUM {
  RLX_F32 = 0, RLX_BF16 = 1, RLX_F16 = 2, RLX_I8 = 3, RLX_U4X2 = 4, RLX_I32 = 5, RLX_U8 = 6
} rlx_dtype;

/* The masked-attention primitive's MaskKind (Section III-A): None, Causal,
 * SlidingWindow(w), Custom (an explicit mask). */
typedef RLX_ENUM {
  RLX_MASK_NONE = 0,
  RLX_MASK_CAUSAL = 1,          /* key j visible to query i iff j <= i                */
  RLX_MASK_SLIDING_WINDOW = 2,  /* iff i - window < j <= i                            */
  RLX_MASK_CUSTOM = 3           /* iff key_mask[b][j] != 0 (key_mask required)        */
} rlx_mask_kind;

/* Weight-only quantisation schemes of Op::DequantMatMul (Sections III-A, VI). */
typedef RLX_ENUM {
  RLX_Q_NONE = 0,              /* w has the activation dtype (f32 or bf16), [N,K]      */
  RLX_Q_INT8_PER_CHANNEL = 1,  /* w int8 [N,K]; scales f16 [N]; W = q * s[n]          */
  RLX_Q_INT4_GROUP_ZP = 2,     /* w u8 [N,K/2], two codes per byte (k = 2j in the low
                                  nibble, 2j+1 in the high nibble); scales and zeros
                                  f16 [N, K/group]; W = (q - z[n,g]) * s[n,g],
                                  g = k / group                                       */
  RLX_Q_INT8_GROUP = 3,        /* w int8 [N,K]; scales f16 [N, K/group];
                                  W = q * s[n,g] (GGUF Q8_0 after rlx_gguf_repack)    */
  RLX_Q_INT4_GROUP_MIN = 4,    /* w as RLX_Q_INT4_GROUP_ZP; `zeros` holds mins m, f16
                                  [N, K/group]; W = q * s[n,g] + m[n,g]
                                  (GGUF Q4_1 and Q4_K after rlx_gguf_repack)         */
  RLX_Q_INT8_GROUP16 = 5       /* w int8 [N,K]; scales f16 [N, K/16]; group_size 16;
                                  W = q * s[n, k/16] (GGUF Q6_K after rlx_gguf_repack) */
} rlx_quant;

typedef RLX_ENUM {
  RLX_EPI_NONE = 0,           /* y = acc                                   */
  RLX_EPI_BIAS = 1,           /* y = acc + bias[n]                         */
  RLX_EPI_BIAS_GELU = 2,      /* y = GELU(acc + bias[n]), erf form         */
  RLX_EPI_BIAS_RESIDUAL = 3   /* y = acc + bias[n] + residual[m][n]        */
} rlx_epilogue;

/* ------------------------------------------------------------------------ */
/* Masked multi-head attention (Section III-A: attention with an explicit
 * MaskKind; Section III-B: Q, K and V read as strided narrows of one buffer).
 *
 * For every sequence b < B, head h < num_heads, query i < S:
 *   out[b,i,h,:] = sum_j P_ij v[b,j,h,:],  P_i = softmax over visible j of
 *                  scale * <q[b,i,h,:], k[b,j,h,:]>
 * with visibility given by `kind` (see rlx_mask_kind) and, when key_mask is
 * non-NULL, additionally key_mask[b*S + j] != 0.  A query with no visible key
 * gets an all-zero output row.
 *
 * Layout: element (b, s, h, d) of q, k and v is at
 *   ptr[(b*S + s) * qkv_row_stride + h*head_dim + d]
 * so q, k, v may be column offsets into one fused [B*S, 3*H] projection
 * (stride 3*H) or separate [B*S, H] tensors (stride H); out is
 *   out[(b*S + s) * out_row_stride + h*head_dim + d].
 * dt: RLX_BF16 (fp32 softmax and accumulation, output rounded to bf16) or
 * RLX_F32.  key_mask: u8 [B,S] or NULL (required for RLX_MASK_CUSTOM).
 * window >= 1 for RLX_MASK_SLIDING_WINDOW, ignored otherwise.
 * Supported: head_dim == 32; 1 <= S <= 512; qkv_row_stride and
 * out_row_stride multiples of 8 and >= num_heads*head_dim; q, k, v, out
 * 16-byte aligned.  Otherwise RLX_ERR_UNSUPPORTED.
 */
rlx_status rlx_masked_attention(const void* q, const void* k, const void* v, int64_t qkv_row_stride,
                                void* out, int64_t out_row_stride, int B, int S, int num_heads, int head_dim,
                                rlx_dtype dt, rlx_mask_kind kind, const uint8_t* key_mask, int window,
                                float scale, void* stream);

/* ------------------------------------------------------------------------ */
/* Matrix multiply with weights dequantised on the fly and a fused epilogue
 * (Op::DequantMatMul, Sections III-A and VI; Linear block, Section III-A):
 *
 *   y[m,n] = epi( sum_k x[m,k] * W[n,k] )      0 <= m < M, 0 <= n < N
 *
 * x: [M,K] row-major, dtype x_dt (RLX_BF16 or RLX_F32; quantised schemes
 * need RLX_BF16).  W: [N,K] in the layout of `scheme` (nn.Linear
 * convention: one row per output feature).  bias: f32 [N] (needed by every
 * epilogue except RLX_EPI_NONE).  y: [M,N] of dtype y_dt: RLX_BF16 or
 * RLX_F32 for bf16 x, RLX_F32 for f32 x.  residual: [M,N] of dtype y_dt
 * (only for RLX_EPI_BIAS_RESIDUAL).  Accumulation is fp32; bf16 outputs are
 * rounded once at the end, f32 outputs are the fp32 result of the epilogue.
 * int8: the integer codes enter the bf16 matrix cores exactly and the
 * per-channel scale is applied to the fp32 sum.  int4: each weight
 * (q - z) * s is formed in fp32 and rounded to bf16 before the product,
 * except in the few-row path below.
 * Few rows (the GEMV regime: 1 <= M <= 16, quantised weights, K a multiple
 * of 128, M * K * 2 <= 65536, scales and zeros 4-byte aligned) take a
 * dedicated kernel that streams the weights once: int8 per-channel as above;
 * no group-scheme weight is rounded: per group, int8 group (32 or 16 k)
 * gives s * sum_k x_k q_k, int4 s * (sum_k x_k (128 + q_k) - (128 + z) sum_k x_k),
 * int4 min s * sum_k x_k (128 + q_k) + (m - 128 s) sum_k x_k, all in fp32.  Results of both paths are deterministic (the same
 * inputs give the same bits), and a row's result does not depend on the
 * other rows of the call.
 * int8 group: q * s formed in fp32 and rounded to bf16 before the product;
 * int4 min: q * s + m formed in fp32 (one rounding) and rounded to bf16
 * (both except in the few-row path below).
 * Supported: M >= 0 (M == 0 is a no-op), N and K positive multiples of 64,
 * group_size == 32 for the group schemes (16 for RLX_Q_INT8_GROUP16;
 * ignored for int8 per-channel),
 * 16-byte aligned x, w, residual and y; y_dt as above.  Otherwise
 * RLX_ERR_UNSUPPORTED.
 */
rlx_status rlx_dequant_matmul(const void* x, rlx_dtype x_dt, int M, int K, const void* w, rlx_quant scheme,
                              const void* scales, const void* zeros, int group_size, int N,
                              const float* bias, const void* residual, rlx_epilogue epi, void* y,
                              rlx_dtype y_dt, void* stream);

/* Test support for the dequantisation step alone: writes the dequantised
 * weights W[n,k] as f32 [N,K] (products of a code and an f16 scale are exact
 * in fp32; q * s + m of int4 min is rounded once, by a fused multiply-add).
 * Same weight layouts and limits as rlx_dequant_matmul;
 * scheme must not be RLX_Q_NONE.
 */
rlx_status rlx_dequant_unpack(const void* w, rlx_quant scheme, const void* scales, const void* zeros,
                              int group_size, int N, int K, float* w_out, void* stream);

/* GGUF weight blocks (the llama.cpp scheme set of Op::DequantMatMul, Section
 * VI).  A tensor of N rows of K weights is N * K/32 consecutive 32-weight
 * blocks (K-quants: N * K/256 super-blocks of 256 weights), row-major; the
 * tensor type ids and blocks are GGUF's:
 *   RLX_GGUF_Q4_0  18 bytes: f16 d, 16 bytes of nibbles   W = (q - 8) * d
 *   RLX_GGUF_Q4_1  20 bytes: f16 d, f16 m, 16 bytes        W = q * d + m
 *   RLX_GGUF_Q8_0  34 bytes: f16 d, 32 int8                W = q * d
 *   RLX_GGUF_Q4_K 144 bytes: f16 d, f16 dmin, 12 bytes of 6-bit sub-block
 *                  scales sc_j and mins mn_j, 128 bytes of nibbles
 *                                                          W = d sc_j q - dmin mn_j
 *   RLX_GGUF_Q6_K 210 bytes: 128 bytes of low nibbles, 64 bytes of high bit
 *                  pairs, 16 int8 sub-block scales sc_i, f16 d
 *                                                          W = d sc_i (q - 32)
 * (4-bit blocks: element j < 16 in the low nibble of byte j, element j + 16
 * in its high nibble; Q4_K / Q6_K: sub-blocks of 32 / 16 weights in the
 * published bit layouts; f16 little-endian).
 * rlx_gguf_repack rewrites such a tensor, once, into the layout of an
 * rlx_quant scheme, and stores that scheme in *scheme (if non-NULL):
 *   Q4_0 -> RLX_Q_INT4_GROUP_ZP  (codes [N,K/2], scales = d, zeros = 8)
 *   Q4_1 -> RLX_Q_INT4_GROUP_MIN (codes [N,K/2], scales = d, zeros = m)
 *   Q8_0 -> RLX_Q_INT8_GROUP     (codes [N,K] int8, scales = d; zeros unused)
 *   Q4_K -> RLX_Q_INT4_GROUP_MIN (codes [N,K/2], scales = f16(d sc_j),
 *                                 zeros = f16(0 - dmin mn_j))
 *   Q6_K -> RLX_Q_INT8_GROUP16   (codes [N,K] int8 = q - 32, scales =
 *                                 f16(d sc_i) [N, K/16]; zeros unused)
 * The basic blocks map exactly.  A K-quant's composed sub-block scales and
 * mins have up to 17 (Q4_K) / 19 (Q6_K) significant bits and are rounded once
 * to f16 (nearest even): the repacked weights are within 2^-11 (|s q| + |m|)
 * of the format's values, and the composed values must be finite in f16.
 * scales and zeros are f16 [N, K/32] (Q6_K: scales [N, K/16]).  Pass the
 * results to rlx_dequant_matmul with group_size 32 (Q6_K: 16).  Device
 * pointers owned by the caller; blocks, scales and zeros 2-byte aligned,
 * codes 16-byte aligned; K a positive multiple of 64 (K-quants: of 256),
 * N >= 0 (N == 0 is a no-op).  Otherwise RLX_ERR_UNSUPPORTED (type,
 * alignment, K) or RLX_ERR_INVALID_ARG.
 */
typedef RLX_ENUM {
  RLX_GGUF_Q4_0 = 2, RLX_GGUF_Q4_1 = 3, RLX_GGUF_Q8_0 = 8, RLX_GGUF_Q4_K = 12, RLX_GGUF_Q6_K = 14
} rlx_gguf_type;

rlx_status rlx_gguf_repack(const void* blocks, rlx_gguf_type type, int N, int K, void* codes, void* scales,
                           void* zeros, rlx_quant* scheme, void* stream);

/* ------------------------------------------------------------------------ */
/* Block-scaled minifloat matmul (the ScaledMatMul path of Section VI:
 * block-scaled FP8 / FP6 / FP4 minifloats, checked bit for bit against an
 * F32 reference), with the OCP Microscaling (MX v1.0) element formats:
 *
 *   y[m,n] = sum_k X(m,k) * W(n,k),   0 <= m < M, 0 <= n < N
 *   X(m,k) = 2^(x_scales[m*K/32 + k/32] - 127) * decode_fx(code of x at (m,k)),
 *   W(n,k) likewise (nn.Linear convention: one W row per output column).
 *
 * Element formats (rlx_mx_format): E4M3 and E5M2 (one byte per code), E2M3
 * and E3M2 (four codes per three bytes: code i of a row occupies bits
 * 6i .. 6i+5 of the row's bytes read as one little-endian integer), E2M1
 * (two codes per byte, the lower k in the low nibble).  Every row of x is
 * K*bits/8 bytes, rows contiguous; likewise w.  Scales: one E8M0 byte per
 * row and 32-element block, [M, K/32] and [N, K/32].  y: f32 [M, N].
 * The products are exact and the sums are accumulated in fp32 by the matrix
 * cores, which add the 64 products of one instruction with a narrow aligned
 * adder: the result is bit-exact when the products of each 64-element step
 * are close in magnitude and every partial sum is exact in fp32; otherwise its
 * error stays below 2^-10 * sum_k |X(m,k) W(n,k)| (measured: 2^-11.3).
 * NaN / Inf codes and the NaN scale (255) give unspecified results.
 * Supported: M >= 0 (M == 0 is a no-op; x, x_scales and y may then be
 * NULL), N and K positive multiples of 128;
 * x, w and y 16-byte aligned, x_scales and w_scales 4-byte aligned.
 * Otherwise RLX_ERR_UNSUPPORTED (alignment, sizes) or RLX_ERR_INVALID_ARG.
 * All pointers are device pointers owned by the caller.
 */
typedef RLX_ENUM { RLX_MX_E4M3 = 0, RLX_MX_E5M2 = 1, RLX_MX_E2M3 = 2, RLX_MX_E3M2 = 3, RLX_MX_E2M1 = 4 } rlx_mx_format;

rlx_status rlx_scaled_matmul(const void* x, const uint8_t* x_scales, rlx_mx_format fx, const void* w,
                             const uint8_t* w_scales, rlx_mx_format fw, int M, int N, int K, float* y,
                             void* stream);

/* ------------------------------------------------------------------------ */
/* Encoder: compile once (bind weights, plan the workspace), run many times
 * (the paper's Session::compile -> CompiledGraph executed with bound inputs,
 * Section III-C).
 */
typedef RLX_ENUM { RLX_INPUT_IDS = 0, RLX_INPUT_HIDDEN = 1 } rlx_input_kind;
typedef RLX_ENUM { RLX_OUTPUT_POOLED = 0, RLX_OUTPUT_HIDDEN = 1 } rlx_output_kind;

typedef struct {
  int hidden;        /* H = heads * head_dim (384)                        */
  int heads;         /* 12                                               */
  int head_dim;      /* 32 (only supported value)                        */
  int ffn;           /* F (1536)                                         */
  int layers;        /* >= 1                                             */
  int vocab;         /* word-embedding rows (IDS input)                  */
  int max_pos;       /* position-embedding rows; >= max_seq (IDS input)  */
  int type_vocab;    /* token-type rows (>= 1, row 0 is used)            */
  float ln_eps;      /* LayerNorm epsilon (1e-12)                        */
  rlx_dtype dtype;   /* RLX_F32 or RLX_BF16: activations, tables, unquantised weights */
  rlx_quant quant;   /* linear-weight scheme; quantised needs RLX_BF16   */
  int group_size;    /* 32 for RLX_Q_INT4_GROUP_ZP                       */
  rlx_input_kind input_kind;
  rlx_output_kind output_kind;
  int max_batch;     /* <= 8192; workspace is planned for max_batch * max_seq tokens */
  int max_seq;       /* <= 512                                           */
  int use_graph;     /* 1: record each (B,S,buffers) forward once as a HIP graph and replay it;
                        0: launch the kernels one by one.  On MI355X the two measure within
                        about 2% of each other for this forward, either one ahead from run
                        to run (the launches hide behind the running kernels) */
} rlx_encoder_config;

/* One layer's weights.  Linear weights follow the nn.Linear convention
 * ([out,in]); their dtype is the config's dtype when quant is RLX_Q_NONE,
 * otherwise the scheme's layout (see rlx_quant), with *_scales / *_zeros
 * pointing at the f16 scale / zero-point arrays (NULL when unused).
 * wqkv stacks the Q, K and V projections: rows [0,H) Q, [H,2H) K, [2H,3H) V;
 * head h owns rows h*head_dim .. h*head_dim+head_dim-1 of each block.
 * Biases and LayerNorm parameters are f32 and 16-byte aligned.
 */
typedef struct {
  const void* wqkv; const void* wqkv_scales; const void* wqkv_zeros; const float* bqkv;  /* [3H,H], [3H] */
  const void* wo;   const void* wo_scales;   const void* wo_zeros;   const float* bo;    /* [H,H],  [H]  */
  const float* ln1_gamma; const float* ln1_beta;                                         /* [H]          */
  const void* w1;   const void* w1_scales;   const void* w1_zeros;   const float* b1;    /* [F,H],  [F]  */
  const void* w2;   const void* w2_scales;   const void* w2_zeros;   const float* b2;    /* [H,F],  [H]  */
  const float* ln2_gamma; const float* ln2_beta;                                         /* [H]          */
} rlx_layer_weights;

typedef struct {
  const void* word_emb;  /* [vocab, H] dtype (IDS input only) */
  const void* pos_emb;   /* [max_pos, H] dtype                 */
  const void* type_emb;  /* [type_vocab, H] dtype              */
  const float* emb_ln_gamma;  /* [H] */
  const float* emb_ln_beta;   /* [H] */
  const rlx_layer_weights* layers;  /* host array of cfg->layers entries; copied by create */
} rlx_encoder_weights;

typedef struct rlx_encoder rlx_encoder;

/* Validates cfg and the weight pointers, allocates the workspace for
 * max_batch * max_seq tokens on the current HIP device, and returns a handle
 * in *out.  `cfg` and `w` are host pointers; they are copied.
 * With dense bf16 weights (quant RLX_Q_NONE) and hidden a multiple of 128,
 * the forward applies each post-LN LayerNorm in the kernels that read its
 * output (Section VIII-B's encoder, same result up to rounding): create then
 * derives, synchronously, copies of w1 of every layer and wqkv of layers
 * 1.. with the preceding LayerNorm's gamma folded in, and folded biases from
 * beta, bqkv and b1; later changes to those arrays, the LayerNorm parameters
 * or bqkv/b1 are not seen by the handle.
 * With quantised weights (bf16 activations) and pooled output, the handle
 * also holds bf16 copies of every layer's matrices (Section VI's
 * DequantMatMul, taken once per forward): the first kernel of each forward
 * dequantises all layers into them, with the gamma fold above, and the rest
 * of the forward runs the dense bf16 kernels (the folded vectors come from
 * the codes, scales and LayerNorm parameters at create, so the weights must
 * keep their values).  RLX_DEQUANT_PROLOGUE_MIN_TOKENS=<n> in the environment at
 * create makes only calls with B * S >= n take it and the others run the
 * dequantising GEMMs (n < 0: never); by default every call takes it.
 * Quantised weights with hidden-state output run the dequantising GEMMs with
 * LayerNorm kernels.
 * Errors: RLX_ERR_INVALID_ARG (nulls, non-positive sizes, H != heads*head_dim),
 * RLX_ERR_UNSUPPORTED (head_dim != 32, H or F not a multiple of 64,
 * max_seq > 512 or > max_pos, quantised weights with f32 activations,
 * group_size != 32, biases or LayerNorm parameters not 16-byte aligned),
 * RLX_ERR_OOM, RLX_ERR_HIP. */
rlx_status rlx_encoder_create(const rlx_encoder_config* cfg, const rlx_encoder_weights* w, rlx_encoder** out);

/* One forward pass.
 * input: IDS -> int32 ids [B,S] in [0, vocab); HIDDEN -> [B,S,H] of cfg.dtype.
 * attention_mask: u8 [B,S], 1 = real token.  Masked tokens are excluded as
 * attention keys, from pooling, and produce zero rows in hidden output.
 * Token (b,s) uses position embedding row s and token-type row 0.
 * output: f32, [B,H] L2-normalised masked-mean embeddings (POOLED) or
 * [B,S,H] final hidden states with zero rows at masked tokens (HIDDEN).
 * Requires 1 <= B <= max_batch, 1 <= S <= max_seq; ids outside the vocabulary
 * are clamped to row vocab-1 rather than read out of bounds.
 * The handle's workspace is reused: do not run two forwards of one handle
 * concurrently on different streams. */
rlx_status rlx_encoder_forward(rlx_encoder* enc, const void* input, const uint8_t* attention_mask, int B, int S,
                               void* output, void* stream);

/* The same forward without a handle and without allocating anything, for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  cfg and w are as for
 * rlx_encoder_create (host pointers, read during the call; the weights are
 * device pointers), input / attention_mask / output as for
 * rlx_encoder_forward, with B and S the only size limits that apply
 * (cfg->max_batch, max_seq and use_graph are ignored).  The workspace (token
 * maps and activations) lives in a static 16 MiB array that the library holds
 * on each GPU it runs on until the process ends: B * S tokens must fit it --
 * about 1900 bf16 or 950 f32 tokens at hidden 384, ffn 1536 -- otherwise
 * RLX_ERR_UNSUPPORTED.  The LayerNorms run as separate kernels (the handle's
 * forward folds them into weights derived at create time), so results agree
 * with rlx_encoder_forward up to rounding.  Every call on one GPU uses that
 * GPU's one array: calls that overlap on one GPU (concurrent streams or host
 * threads) race and must be serialised by the caller.  Errors as for
 * rlx_encoder_create and rlx_encoder_forward. */
rlx_status rlx_encoder_forward_noalloc(const rlx_encoder_config* cfg, const rlx_encoder_weights* w,
                                       const void* input, const uint8_t* attention_mask, int B, int S, void* output,
                                       void* stream);

/* Frees the workspace and cached graphs after waiting for the last forward
 * enqueued through the handle (an event recorded on its stream) -- not for
 * the rest of the device.  NULL is ignored. */
void rlx_encoder_destroy(rlx_encoder* enc);

/* Forward passes with dense bf16 weights, id input, pooled output, hidden
 * 384 (heads of 32), FFN a multiple of 128, at most 12 layers, and per call
 * B <= 256, S <= 128, B * S <= 32768, run as one persistent launch: resident
 * blocks, each XCD working on its own run of sequences, every tile starting
 * when the tiles it reads are done.  rlx_encoder_create selects it when
 * RLX_PIPELINE=1 is set in the environment (otherwise forwards launch one
 * kernel per step).  Same results up to rounding.
 * Returns 1 when the handle's supported forwards take the persistent launch. */
int rlx_encoder_uses_persistent_forward(const rlx_encoder* enc);

/* Waits for the last forward enqueued through the handle, then reports
 * whether a wait inside the persistent launch of it or of an earlier forward
 * gave up (bounded waits: after ~0.5 s without progress the launch finishes
 * with invalid outputs instead of hanging): RLX_ERR_HIP with a message, after
 * which the report is cleared.  RLX_OK otherwise (always for handles without
 * the persistent launch). */
rlx_status rlx_encoder_check(rlx_encoder* enc);

/* Per-kernel timing of forward passes (a native counterpart of a per-operator
 * dispatch report).  While enabled, each forward runs normally, then replays,
 * kernel by kernel in forward order, a HIP graph holding 8 back-to-back
 * launches of that kernel alone between two HIP events, and finally runs the
 * forward again, so the output is the forward's result; the call is then
 * synchronous.  Each kernel adds one launch and its mean time per launch to
 * its class.  rlx_encoder_profile_read returns, for every class with launches,
 * the number of launches and the summed time in milliseconds, then clears the
 * totals.  Names are static strings owned by the library. */
rlx_status rlx_encoder_set_profiling(rlx_encoder* enc, int enable);
rlx_status rlx_encoder_profile_read(rlx_encoder* enc, int max_entries, const char** names, int* launches,
                                    double* total_ms, int* n_entries);

/* Test support for token compaction, the index work a forward starts with
 * (Section VIII-B's inputs are padded batches; every later kernel of a
 * forward runs on the real tokens only).  This is the kernel a forward runs
 * for hidden-state input and for masks of more than 16384 entries; the
 * embedding kernel computes the same maps itself for smaller masks.
 * From attention_mask u8 [B,S] (nonzero = real token) it writes, to int32
 * device arrays owned by the caller:
 *   cu [B+1]       cu[b] = the number of real tokens of sequences 0 .. b-1;
 *   tok_src [B*S]  entries 0 .. cu[B]-1: b*S + s of every real token,
 *                  sequences in order, positions ascending (the entries after
 *                  them are not written);
 *   tok_dst [B*S]  the index of token (b,s) in tok_src, or -1 when masked;
 *   order [B]      (NULL skips it; requires B <= 256) the sequences by
 *                  real-token count, longest first, ties by sequence index.
 * Requires 1 <= B <= 8192 and 1 <= S <= 512 (RLX_ERR_UNSUPPORTED beyond),
 * non-null mask, cu, tok_src and tok_dst (RLX_ERR_INVALID_ARG). */
rlx_status rlx_mask_compaction(const uint8_t* attention_mask, int B, int S, int32_t* cu, int32_t* tok_src,
                               int32_t* tok_dst, int32_t* order, void* stream);

/* Test support: copies the token compaction maps that the handle's most
 * recent forward computed (layouts as for rlx_mask_compaction, for that
 * forward's B and S, which must be the ones passed: RLX_ERR_INVALID_ARG
 * otherwise) into caller-owned int32 device arrays.  The copies are enqueued
 * on `stream`; order them after the forward.  order (NULL skips it) requires
 * B <= 256.  Handles that take the persistent forward keep no maps
 * (RLX_ERR_UNSUPPORTED). */
rlx_status rlx_encoder_token_maps(const rlx_encoder* enc, int B, int S, int32_t* cu, int32_t* tok_src,
                                  int32_t* tok_dst, int32_t* order, void* stream);

/* Message describing the last error on the calling thread ("" if none).
 * Valid until the next rlx_* call on this thread. */
const char* rlx_last_error(void);

/* Library version string, e.g. "rlx-mi355x 0.1.0 (gfx950)". */
const char* rlx_version(void);

#ifdef __cplusplus
}
#endif
#endif /* RLX_H_ */
