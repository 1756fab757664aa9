// C ABI: argument validation, the encoder handle (bound weights + planned
// workspace + cached HIP graphs), per-kernel profiling and error reporting.
//
// The paper's runtime compiles a graph once for a device and executes the
// cached schedule with bound inputs (Section III-C), and its dispatch fails
// with a diagnostic instead of silently degrading (Section IV).  Here:
// rlx_encoder_create binds the weights and allocates one workspace for
// max_batch * max_seq tokens; rlx_encoder_forward validates everything
// before enqueueing anything, then replays a HIP graph recorded for the same
// (B, S, buffers) or records one.  Unsupported requests return
// RLX_ERR_UNSUPPORTED with a message; no other code path is ever taken.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/rlx.h"
#include "kernels.hpp"

using namespace rlx;

namespace {

thread_local std::string g_last_error;

rlx_status fail(rlx_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

rlx_status ok() {
  g_last_error.clear();
  return RLX_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

rlx_status hip_fail(hipError_t e, const char* what) {
  (void)hipGetLastError();  // the error is reported here; do not leave it for the caller's next HIP call
  return fail(RLX_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define RLX_HIP(call, what)                        \
  do {                                             \
    hipError_t e_ = (call);                        \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

const char* dtype_name(rlx_dtype d) {
  switch (d) {
    case RLX_F32: return "f32";
    case RLX_BF16: return "bf16";
    case RLX_F16: return "f16";
    case RLX_I8: return "i8";
    case RLX_U4X2: return "u4x2";
    case RLX_I32: return "i32";
    case RLX_U8: return "u8";
  }
  return "?";
}

rlx_status check_attention_args(const void* q, const void* k, const void* v, int64_t ld, const void* out,
                                int64_t ld_out, int B, int S, int heads, int head_dim, rlx_dtype dt,
                                rlx_mask_kind kind, const uint8_t* key_mask, int window, float scale) {
  if (B < 0 || S < 0) return fail(RLX_ERR_INVALID_ARG, "attention: B=%d and S=%d must be >= 0", B, S);
  if (heads <= 0 || head_dim <= 0)
    return fail(RLX_ERR_INVALID_ARG, "attention: num_heads=%d and head_dim=%d must be positive", heads, head_dim);
  if (!q || !k || !v || !out) return fail(RLX_ERR_INVALID_ARG, "attention: q, k, v and out must be non-null");
  if (kind < RLX_MASK_NONE || kind > RLX_MASK_CUSTOM)
    return fail(RLX_ERR_INVALID_ARG, "attention: unknown mask kind %d", (int)kind);
  if (kind == RLX_MASK_CUSTOM && !key_mask)
    return fail(RLX_ERR_INVALID_ARG, "attention: RLX_MASK_CUSTOM needs a key mask");
  if (kind == RLX_MASK_SLIDING_WINDOW && window < 1)
    return fail(RLX_ERR_INVALID_ARG, "attention: sliding window %d must be >= 1", window);
  if (!std::isfinite(scale)) return fail(RLX_ERR_INVALID_ARG, "attention: scale must be finite");
  if (dt != RLX_BF16 && dt != RLX_F32)
    return fail(RLX_ERR_UNSUPPORTED, "attention: dtype %s not supported (bf16, f32)", dtype_name(dt));
  if (head_dim != 32) return fail(RLX_ERR_UNSUPPORTED, "attention: head_dim %d not supported (32)", head_dim);
  if (S > 512) return fail(RLX_ERR_UNSUPPORTED, "attention: S=%d exceeds 512", S);
  const int64_t hw = (int64_t)heads * head_dim;
  if (ld < hw || ld_out < hw)
    return fail(RLX_ERR_INVALID_ARG, "attention: row strides (%lld, %lld) smaller than heads*head_dim=%lld",
                (long long)ld, (long long)ld_out, (long long)hw);
  if (ld % 8 || ld_out % 8)
    return fail(RLX_ERR_UNSUPPORTED, "attention: row strides must be multiples of 8 elements");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
    return fail(RLX_ERR_UNSUPPORTED, "attention: q, k, v and out must be 16-byte aligned");
  return RLX_OK;
}

rlx_status check_quant_weights(const char* who, rlx_quant scheme, const void* w, const void* scales,
                               const void* zeros, int group_size, int N, int K) {
  if (!w) return fail(RLX_ERR_INVALID_ARG, "%s: weight pointer is null", who);
  if (scheme < RLX_Q_NONE || scheme > RLX_Q_INT8_GROUP16)
    return fail(RLX_ERR_INVALID_ARG, "%s: unknown quantisation scheme %d", who, (int)scheme);
  if (N % 64 || K % 64)
    return fail(RLX_ERR_UNSUPPORTED, "%s: N=%d and K=%d must be multiples of 64", who, N, K);
  if (!aligned16(w)) return fail(RLX_ERR_UNSUPPORTED, "%s: weights must be 16-byte aligned", who);
  if ((scheme == RLX_Q_INT8_PER_CHANNEL || scheme == RLX_Q_INT8_GROUP || scheme == RLX_Q_INT8_GROUP16) && !scales)
    return fail(RLX_ERR_INVALID_ARG, "%s: int8 weights need scales", who);
  if ((scheme == RLX_Q_INT4_GROUP_ZP || scheme == RLX_Q_INT4_GROUP_MIN) && (!scales || !zeros))
    return fail(RLX_ERR_INVALID_ARG, "%s: int4 weights need scales and zeros (or mins)", who);
  if (scheme == RLX_Q_INT8_GROUP16 && group_size != 16)
    return fail(RLX_ERR_UNSUPPORTED, "%s: RLX_Q_INT8_GROUP16 takes group size 16, not %d", who, group_size);
  if (scheme >= RLX_Q_INT4_GROUP_ZP && scheme != RLX_Q_INT8_GROUP16 && group_size != 32)
    return fail(RLX_ERR_UNSUPPORTED, "%s: group size %d not supported (32)", who, group_size);
  return RLX_OK;
}

Quant to_quant(rlx_quant q) {
  switch (q) {
    case RLX_Q_INT8_PER_CHANNEL: return Quant::Int8;
    case RLX_Q_INT4_GROUP_ZP: return Quant::Int4;
    case RLX_Q_INT8_GROUP: return Quant::Int8G;
    case RLX_Q_INT4_GROUP_MIN: return Quant::Int4M;
    case RLX_Q_INT8_GROUP16: return Quant::Int8G16;
    default: return Quant::None;
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// encoder handle
// ---------------------------------------------------------------------------

namespace {

enum KernelClass {
  K_MASK_SCAN = 0, K_EMBED_LN, K_GATHER_ROWS, K_GEMM_QKV, K_ATTENTION, K_GEMM_ATTN_OUT, K_LN1, K_GEMM_FFN_UP,
  K_GEMM_FFN_DOWN, K_LN2, K_POOL, K_SCATTER, K_QKV_ATTENTION, K_PIPE, K_DEQUANT, K_NUM_CLASSES
};
const char* kClassNames[K_NUM_CLASSES] = {"mask_scan",     "embed_ln",    "gather_rows", "gemm_qkv",
                                          "attention",     "gemm_attn_out", "layer_norm_1", "gemm_ffn_up",
                                          "gemm_ffn_down", "layer_norm_2", "pool_l2",     "scatter_hidden",
                                          "qkv_attention", "encoder_pipe", "dequant_weights"};

struct GraphEntry {
  int B, S;
  const void* input;
  const uint8_t* mask;
  void* output;
  hipGraphExec_t exec;
  uint64_t last_use;
};

struct KernelSlot {  // one launch of a forward: its class and a replayable closure
  int cls;
  std::function<hipError_t(hipStream_t)> launch;
};

struct ProfGraph {  // per forward configuration: one graph of kProfReps launches per kernel
  GraphEntry g;
  std::vector<int> slot_cls;
  std::vector<hipGraphExec_t> slot_exec;
};
constexpr int kProfReps = 8;

}  // namespace

struct rlx_encoder {
  rlx_encoder_config cfg;
  rlx_encoder_weights w;
  std::vector<rlx_layer_weights> layers;
  int device = 0;
  DType dt = DType::BF16;
  void* ws = nullptr;
  int* cu = nullptr;
  int* tok_src = nullptr;
  int* tok_dst = nullptr;
  int* order = nullptr;  // sequences by token count, longest first (mask scan, B <= kMaxOrderedBatch)
  int2* rank_rows = nullptr;  // (first row, real tokens) of order[r] at entry r (written with the order)
  int last_B = 0, last_S = 0;  // shape of the most recent forward (its token maps are in the workspace)
  void *X = nullptr, *X1 = nullptr, *A = nullptr, *CTX = nullptr, *QKV = nullptr, *G = nullptr;
  // Deferred LayerNorm (dense bf16 weights): no kernel writes a LayerNorm
  // output.  The output projection and FFN-down store their pre-norm sums (A,
  // and X from the second layer on) with per-row partial statistics (S1, S2);
  // the kernels that read those rows normalise them.  The QKV projection of
  // layers 1.. and every FFN-up projection take weights with the preceding
  // LayerNorm folded in, derived at create time.
  bool deferred = false;
  float2* S1 = nullptr;  // statistics of A (LN1 input)
  float2* S2 = nullptr;  // statistics of X from the second layer on (LN2 input)
  struct Folded {
    void* wqkv = nullptr; float* uq = nullptr; float* vq = nullptr;  // layers >= 1: LN2 of the previous layer
    void* w1 = nullptr; float* u1 = nullptr; float* v1 = nullptr;    // LN1 of the same layer
  };
  std::vector<Folded> folded;
  void* fold_mem = nullptr;
  // Quantised weights, calls of at least dq_min_tokens = B*S positions: one
  // kernel at the start of the forward dequantises every layer to bf16
  // (gamma folded in where the dense deferred LayerNorm wants it) and the
  // forward runs the bf16 kernels on them (dq_cfg, dq_layers, dq_folded).
  // Smaller calls run the dequantising GEMMs.
  int dq_min_tokens = -1;  // < 0: never
  void* dq_mem = nullptr;  // bf16 weights, folded vectors, then the job table
  const DequantJob* dq_jobs = nullptr;
  int dq_njobs = 0, dq_max_elems = 0;
  rlx_encoder_config dq_cfg{};
  std::vector<rlx_layer_weights> dq_layers;
  std::vector<Folded> dq_folded;
  // Persistent forward (pipe.hip): chosen at create for the shapes it
  // supports; its per-layer pointer table and per-XCD sync words live in
  // pipe_mem.
  bool pipe = false;
  int pipe_grid = 0;
  void* pipe_mem = nullptr;
  PipeLayer* pipe_layers = nullptr;
  int* pipe_sync = nullptr;
  hipStream_t cap_stream = nullptr;
  // recorded after every forward on the caller's stream: destroy and the graph
  // cache wait for it (the handle's own work) instead of the whole device
  hipEvent_t done_ev = nullptr;
  std::vector<GraphEntry> graphs;
  uint64_t use_clock = 0;
  bool profiling = false;
  hipEvent_t prof_ev[2] = {nullptr, nullptr};
  std::vector<ProfGraph> prof_graphs;
  int prof_cnt[K_NUM_CLASSES] = {0};
  double prof_ms[K_NUM_CLASSES] = {0};
};

namespace {

constexpr size_t kMaxGraphs = 16;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// What one forward reads: the configuration, the bound weights and a
// workspace (token maps and activation buffers for up to B*S tokens).  The
// encoder handle owns one; the handle-free forward builds one over the
// library's static scratch.
struct FwdCtx {
  const rlx_encoder_config* cfg;
  const rlx_encoder_weights* w;
  const rlx_layer_weights* layers;
  DType dt;
  int *cu, *tok_src, *tok_dst, *order;
  void *X, *X1, *A, *CTX, *QKV, *G;
  bool deferred;  // dense bf16: LayerNorms applied by the kernels that read their outputs
  float2 *S1, *S2;
  const rlx_encoder::Folded* folded;
  // the persistent forward, when the handle has it (else pipe_grid == 0)
  int pipe_grid;
  const PipeLayer* pipe_layers;
  int* pipe_sync;
  // the weight dequantisation that starts the forward (dq_njobs == 0: none)
  const DequantJob* dq_jobs;
  int dq_njobs, dq_max_elems;
  int2* rank_rows = nullptr;  // [B]: (first row, real tokens) by launch rank, beside the order
};

// The forward of B sequences of S positions: with the dequantisation prologue
// when the handle has one and the call is large enough (cfg then says dense).
FwdCtx ctx_of(const rlx_encoder* e, int B, int S) {
  const bool dq = e->dq_mem && e->dq_min_tokens >= 0 && (long long)B * S >= e->dq_min_tokens;
  return FwdCtx{dq ? &e->dq_cfg : &e->cfg, &e->w, dq ? e->dq_layers.data() : e->layers.data(), e->dt, e->cu,
                e->tok_src, e->tok_dst, e->order, e->X, e->X1, e->A, e->CTX, e->QKV, e->G, e->deferred, e->S1,
                e->S2, dq ? e->dq_folded.data() : e->folded.data(), e->pipe ? e->pipe_grid : 0, e->pipe_layers,
                e->pipe_sync, dq ? e->dq_jobs : nullptr, dq ? e->dq_njobs : 0, dq ? e->dq_max_elems : 0,
                e->rank_rows};
}

// Workspace layout for max_batch sequences of max_seq tokens (256-byte aligned regions).
struct WsPlan {
  size_t cu, src, dst, ord, rr, X, X1, A, C, Q, G, S1, S2, bytes;
};
WsPlan plan_workspace(size_t max_batch, size_t max_seq, size_t H, size_t F, size_t es, bool deferred) {
  const size_t T = max_batch * max_seq;
  WsPlan p{};
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, 256); return o; };
  p.cu = take((max_batch + 1) * sizeof(int));
  p.src = take(T * sizeof(int));
  p.dst = take(T * sizeof(int));
  p.ord = take(max_batch * sizeof(int));
  p.rr = take(max_batch * sizeof(int2));
  p.X = take(T * H * es); p.X1 = take(T * H * es); p.A = take(T * H * es); p.C = take(T * H * es);
  p.Q = take(T * 3 * H * es); p.G = take(T * F * es);
  const size_t stats_bytes = deferred ? T * (H / 64) * sizeof(float2) : 0;
  p.S1 = take(stats_bytes); p.S2 = take(stats_bytes);
  p.bytes = off;
  return p;
}

void bind_workspace(FwdCtx& c, uint8_t* base, const WsPlan& p) {
  c.cu = reinterpret_cast<int*>(base + p.cu);
  c.tok_src = reinterpret_cast<int*>(base + p.src);
  c.tok_dst = reinterpret_cast<int*>(base + p.dst);
  c.order = reinterpret_cast<int*>(base + p.ord);
  c.rank_rows = reinterpret_cast<int2*>(base + p.rr);
  c.X = base + p.X; c.X1 = base + p.X1; c.A = base + p.A; c.CTX = base + p.C; c.QKV = base + p.Q; c.G = base + p.G;
  c.S1 = c.deferred ? reinterpret_cast<float2*>(base + p.S1) : nullptr;
  c.S2 = c.deferred ? reinterpret_cast<float2*>(base + p.S2) : nullptr;
}

rlx_status check_config(const rlx_encoder_config* c) {
  if (c->hidden <= 0 || c->heads <= 0 || c->head_dim <= 0 || c->ffn <= 0 || c->layers <= 0)
    return fail(RLX_ERR_INVALID_ARG, "encoder: hidden, heads, head_dim, ffn and layers must be positive");
  if (c->hidden != c->heads * c->head_dim)
    return fail(RLX_ERR_INVALID_ARG, "encoder: hidden %d != heads %d * head_dim %d", c->hidden, c->heads,
                c->head_dim);
  if (c->max_batch <= 0 || c->max_seq <= 0)
    return fail(RLX_ERR_INVALID_ARG, "encoder: max_batch and max_seq must be positive");
  if (c->input_kind != RLX_INPUT_IDS && c->input_kind != RLX_INPUT_HIDDEN)
    return fail(RLX_ERR_INVALID_ARG, "encoder: unknown input kind %d", (int)c->input_kind);
  if (c->output_kind != RLX_OUTPUT_POOLED && c->output_kind != RLX_OUTPUT_HIDDEN)
    return fail(RLX_ERR_INVALID_ARG, "encoder: unknown output kind %d", (int)c->output_kind);
  if (!(c->ln_eps >= 0.0f) || !std::isfinite(c->ln_eps))
    return fail(RLX_ERR_INVALID_ARG, "encoder: ln_eps must be finite and >= 0");
  if (c->input_kind == RLX_INPUT_IDS && (c->vocab <= 0 || c->max_pos <= 0 || c->type_vocab <= 0))
    return fail(RLX_ERR_INVALID_ARG, "encoder: vocab, max_pos and type_vocab must be positive for id input");
  if (c->dtype != RLX_F32 && c->dtype != RLX_BF16)
    return fail(RLX_ERR_UNSUPPORTED, "encoder: dtype %s not supported (f32, bf16)", dtype_name(c->dtype));
  if (c->quant < RLX_Q_NONE || c->quant > RLX_Q_INT8_GROUP16)
    return fail(RLX_ERR_INVALID_ARG, "encoder: unknown quantisation scheme %d", (int)c->quant);
  if (c->quant != RLX_Q_NONE && c->dtype != RLX_BF16)
    return fail(RLX_ERR_UNSUPPORTED, "encoder: quantised weights need bf16 activations");
  if (c->quant == RLX_Q_INT8_GROUP16 && c->group_size != 16)
    return fail(RLX_ERR_UNSUPPORTED, "encoder: RLX_Q_INT8_GROUP16 takes group size 16, not %d", c->group_size);
  if (c->quant >= RLX_Q_INT4_GROUP_ZP && c->quant != RLX_Q_INT8_GROUP16 && c->group_size != 32)
    return fail(RLX_ERR_UNSUPPORTED, "encoder: group size %d not supported (32)", c->group_size);
  if (c->head_dim != 32) return fail(RLX_ERR_UNSUPPORTED, "encoder: head_dim %d not supported (32)", c->head_dim);
  if (c->hidden % 64 || c->ffn % 64 || c->hidden > 1024)
    return fail(RLX_ERR_UNSUPPORTED, "encoder: hidden %d and ffn %d must be multiples of 64, hidden <= 1024",
                c->hidden, c->ffn);
  if (c->max_seq > 512) return fail(RLX_ERR_UNSUPPORTED, "encoder: max_seq %d exceeds 512", c->max_seq);
  if (c->input_kind == RLX_INPUT_IDS && c->max_seq > c->max_pos)
    return fail(RLX_ERR_UNSUPPORTED, "encoder: max_seq %d exceeds max_pos %d", c->max_seq, c->max_pos);
  if (c->max_batch > 8192) return fail(RLX_ERR_UNSUPPORTED, "encoder: max_batch %d exceeds 8192", c->max_batch);
  if ((int64_t)c->max_batch * c->max_seq > (int64_t)1 << 24)
    return fail(RLX_ERR_UNSUPPORTED, "encoder: max_batch * max_seq exceeds 2^24 tokens");
  return RLX_OK;
}

rlx_status check_weights(const rlx_encoder_config* c, const rlx_encoder_weights* w) {
  if (!w->layers) return fail(RLX_ERR_INVALID_ARG, "encoder: weights->layers is null");
  if (c->input_kind == RLX_INPUT_IDS) {
    if (!w->word_emb || !w->pos_emb || !w->type_emb || !w->emb_ln_gamma || !w->emb_ln_beta)
      return fail(RLX_ERR_INVALID_ARG, "encoder: embedding tables and embedding LayerNorm parameters are required");
  }
  const int H = c->hidden, F = c->ffn;
  for (int l = 0; l < c->layers; ++l) {
    const rlx_layer_weights& L = w->layers[l];
    if (!L.bqkv || !L.bo || !L.b1 || !L.b2 || !L.ln1_gamma || !L.ln1_beta || !L.ln2_gamma || !L.ln2_beta)
      return fail(RLX_ERR_INVALID_ARG, "encoder: layer %d has a null bias or LayerNorm parameter", l);
    if (!aligned16(L.ln1_gamma) || !aligned16(L.ln1_beta) || !aligned16(L.ln2_gamma) || !aligned16(L.ln2_beta))
      return fail(RLX_ERR_UNSUPPORTED, "encoder: layer %d LayerNorm parameters must be 16-byte aligned", l);
    struct { const char* nm; const void *w, *s, *z; int N, K; const float* b; } lin[4] = {
        {"wqkv", L.wqkv, L.wqkv_scales, L.wqkv_zeros, 3 * H, H, L.bqkv},
        {"wo", L.wo, L.wo_scales, L.wo_zeros, H, H, L.bo},
        {"w1", L.w1, L.w1_scales, L.w1_zeros, F, H, L.b1},
        {"w2", L.w2, L.w2_scales, L.w2_zeros, H, F, L.b2}};
    for (auto& x : lin) {
      char who[64];
      snprintf(who, sizeof who, "encoder layer %d %s", l, x.nm);
      rlx_status st = check_quant_weights(who, c->quant, x.w, x.s, x.z, c->group_size, x.N, x.K);
      if (st != RLX_OK) return st;
      if (!aligned16(x.b)) return fail(RLX_ERR_UNSUPPORTED, "%s: bias must be 16-byte aligned", who);
    }
  }
  return RLX_OK;
}

// Enqueue one forward on `s`.  With `slots` non-null every launch is also
// recorded (kernel class + a closure holding a copy of its arguments) so that
// the profiling mode can replay single kernels.
rlx_status enqueue_forward(const FwdCtx& fc, const void* input, const uint8_t* mask, int B, int S, void* output,
                           hipStream_t s, std::vector<KernelSlot>* slots) {
  // (held by value: a profiled forward's recorded launches copy it and outlive fc)
  const FwdCtx E = fc;
  const rlx_encoder_config& c = *E.cfg;
  const int H = c.hidden, F = c.ffn, T = B * S;
  const int* n_dev = E.cu + B;  // number of real tokens, written by the mask scan
  // Each launch runs at once; only a profiled forward also keeps a replayable
  // closure of it (so a plain forward builds no std::function).
#define STEP(cls, expr)                                                                    \
  do {                                                                                     \
    const hipError_t err_ = [&](hipStream_t ss) -> hipError_t { return (expr); }(s);     \
    if (err_ != hipSuccess) return hip_fail(err_, kClassNames[cls]);                       \
    if (slots) slots->push_back({cls, [=](hipStream_t ss) -> hipError_t { return (expr); }}); \
  } while (0)

  if (E.dq_njobs > 0)  // quantised weights of every layer to bf16 (the rest of the forward is dense)
    STEP(K_DEQUANT, launch_dequant_jobs(E.dq_jobs, E.dq_njobs, E.dq_max_elems, ss));
  if (E.pipe_grid > 0 && pipe_supported(PipeShape{B, S, H, F, c.heads, c.layers})) {
    // the whole forward in one persistent launch (pipe.hip)
    PipeParams pp{};
    pp.mask = mask; pp.ids = static_cast<const int*>(input); pp.B = B; pp.S = S;
    pp.word = static_cast<const bf16_t*>(E.w->word_emb); pp.pos = static_cast<const bf16_t*>(E.w->pos_emb);
    pp.type = static_cast<const bf16_t*>(E.w->type_emb); pp.emb_g = E.w->emb_ln_gamma; pp.emb_b = E.w->emb_ln_beta;
    pp.vocab = c.vocab; pp.eps = c.ln_eps; pp.scale = 1.0f / std::sqrt((float)c.head_dim);
    pp.layers = E.pipe_layers; pp.L = c.layers; pp.H = H; pp.F = F; pp.heads = c.heads;
    pp.X = static_cast<bf16_t*>(E.X); pp.A = static_cast<bf16_t*>(E.A); pp.CTX = static_cast<bf16_t*>(E.CTX);
    pp.G = static_cast<bf16_t*>(E.G); pp.S1 = E.S1; pp.S2 = E.S2; pp.ctx_rows = T;
    pp.last_g = E.layers[c.layers - 1].ln2_gamma; pp.last_b = E.layers[c.layers - 1].ln2_beta;
    pp.out = static_cast<float*>(output); pp.sync = E.pipe_sync;
    const int grid = E.pipe_grid;
    STEP(K_PIPE, launch_encoder_pipe(pp, grid, ss));
    return RLX_OK;
  }
  if (c.input_kind == RLX_INPUT_IDS && embed_scan_supported(B, S)) {
    // small masks: the scan runs inside the embedding kernel
    STEP(K_EMBED_LN, launch_embed_scan(mask, static_cast<const int*>(input), B, S, E.w->word_emb, E.w->pos_emb,
                                       E.w->type_emb, E.w->emb_ln_gamma, E.w->emb_ln_beta, c.ln_eps, c.vocab, H,
                                       E.cu, E.tok_src, E.tok_dst, E.order, E.X, E.dt, ss, E.rank_rows));
  } else {
    STEP(K_MASK_SCAN, launch_mask_scan(mask, B, S, E.cu, E.tok_src, E.tok_dst, E.order, ss, E.rank_rows));
    if (c.input_kind == RLX_INPUT_IDS) {
      STEP(K_EMBED_LN, launch_embed_ln(static_cast<const int*>(input), E.w->word_emb, E.w->pos_emb, E.w->type_emb,
                                       E.w->emb_ln_gamma, E.w->emb_ln_beta, c.ln_eps, c.vocab, S, H, E.tok_src,
                                       n_dev, T, E.X, E.dt, ss));
    } else {
      STEP(K_GATHER_ROWS, launch_gather_rows(input, H, E.tok_src, n_dev, T, E.X, E.dt, ss));
    }
  }
  for (int l = 0; l < c.layers; ++l) {
    const rlx_layer_weights& L = E.layers[l];
    // From the second layer on, a deferred-LayerNorm forward's layer input X
    // holds the previous layer's LN2 input, normalised by its readers.
    const bool x_def = E.deferred && l > 0;
    const rlx_layer_weights* prev = l > 0 ? &E.layers[l - 1] : nullptr;
    const Quant q = to_quant(c.quant);
    // quantised weights keep their codes; their deferred LN inputs are gamma-scaled
    const bool gsc = E.deferred && q != Quant::None;
    const void* wqkv = x_def && !gsc ? E.folded[l].wqkv : L.wqkv;
    const float* bqkv = x_def ? E.folded[l].vq : L.bqkv;
    const float* uqkv = x_def ? E.folded[l].uq : nullptr;
    GemmParams g{};
    g.m_dev = n_dev;
    g.M = T;
    g.dtype = E.dt;
    g.quant = q;
    g.ln_eps = c.ln_eps;

    const bool fused_attn = E.dt == DType::BF16 && q == Quant::None && S <= 128;
    if (fused_attn) {
      FusedAttnParams fa{};
      fa.x = E.X; fa.wqkv = wqkv; fa.bqkv = bqkv; fa.cu_seqlens = E.cu; fa.out = E.CTX; fa.out_rows = T;
      fa.B = B; fa.H = H; fa.heads = c.heads; fa.scale = 1.0f / std::sqrt((float)c.head_dim);
      fa.seq_order = B <= kMaxOrderedBatch ? E.order : nullptr;  // written by the mask scan
      fa.rank_rows = B <= kMaxOrderedBatch ? E.rank_rows : nullptr;  // (with the order)
      fa.x_stats = x_def ? E.S2 : nullptr; fa.fold_u = uqkv; fa.ln_eps = c.ln_eps;
      STEP(K_QKV_ATTENTION, launch_qkv_attention(fa, ss));
    } else {
      g.x = E.X; g.w = wqkv; g.scales = L.wqkv_scales; g.zeros = L.wqkv_zeros; g.bias = bqkv;
      g.residual = nullptr; g.y = E.QKV; g.N = 3 * H; g.K = H; g.epi = Epi::Bias;
      g.x_stats = x_def ? E.S2 : nullptr; g.fold_u = uqkv;
      STEP(K_GEMM_QKV, launch_gemm(g, ss));
      g.x_stats = nullptr; g.fold_u = nullptr;

      AttnParams a{};
      const size_t es = E.dt == DType::BF16 ? 2 : 4;
      a.q = E.QKV;
      a.k = static_cast<const uint8_t*>(E.QKV) + (size_t)H * es;
      a.v = static_cast<const uint8_t*>(E.QKV) + (size_t)2 * H * es;
      a.ld_qkv = 3 * H;
      a.out = E.CTX; a.ld_out = H;
      a.B = B; a.S = S; a.heads = c.heads; a.kind = 0; a.key_mask = nullptr; a.window = 0;
      a.scale = 1.0f / std::sqrt((float)c.head_dim);
      a.cu_seqlens = E.cu;
      a.dtype = E.dt;
      STEP(K_ATTENTION, launch_attention(a, ss));
    }

    g.x = E.CTX; g.w = L.wo; g.scales = L.wo_scales; g.zeros = L.wo_zeros; g.bias = L.bo;
    g.residual = E.X; g.y = E.A; g.N = H; g.K = H; g.epi = Epi::BiasResidual;
    g.x_head_rows = fused_attn ? T : 0;  // the fused attention writes the context head-major
    if (x_def) {
      g.res_stats = E.S2; g.res_gamma = prev->ln2_gamma; g.res_beta = prev->ln2_beta; g.res_scaled = gsc;
    }
    g.y_stats = E.deferred ? E.S1 : nullptr;
    g.y_gamma = gsc ? L.ln1_gamma : nullptr;
    STEP(K_GEMM_ATTN_OUT, launch_gemm(g, ss));
    g.x_head_rows = 0;
    g.res_stats = nullptr; g.res_gamma = g.res_beta = nullptr; g.y_stats = nullptr;
    g.res_scaled = false; g.y_gamma = nullptr;

    if (E.deferred) {
      // FFN-up on LN1(A) with LN1 folded into W1; FFN-down's residual LN1(A)
      // is normalised in its epilogue, and its output is LN2's input
      g.x = E.A; g.x_stats = E.S1; g.fold_u = E.folded[l].u1;
      if (gsc) {
        g.w = L.w1; g.scales = L.w1_scales; g.zeros = L.w1_zeros;
      } else {
        g.w = E.folded[l].w1; g.scales = nullptr; g.zeros = nullptr;
      }
      g.bias = E.folded[l].v1;
      g.residual = nullptr; g.y = E.G; g.N = F; g.K = H; g.epi = Epi::BiasGelu;
      STEP(K_GEMM_FFN_UP, launch_gemm(g, ss));
      g.x_stats = nullptr; g.fold_u = nullptr;

      g.x = E.G; g.w = L.w2; g.scales = L.w2_scales; g.zeros = L.w2_zeros; g.bias = L.b2;
      g.residual = E.A; g.res_stats = E.S1; g.res_gamma = L.ln1_gamma; g.res_beta = L.ln1_beta; g.res_scaled = gsc;
      g.y = E.X; g.y_stats = E.S2; g.y_gamma = gsc ? L.ln2_gamma : nullptr; g.N = H; g.K = F;
      g.epi = Epi::BiasResidual;
      STEP(K_GEMM_FFN_DOWN, launch_gemm(g, ss));
      g.res_scaled = false; g.y_gamma = nullptr;
      continue;
    }

    // LN1 feeds the FFN-up projection and, as the residual, the FFN-down one.
    STEP(K_LN1, launch_layer_norm(E.A, L.ln1_gamma, L.ln1_beta, c.ln_eps, H, n_dev, T, E.X1, E.dt, ss));
    g.x = E.X1; g.w = L.w1; g.scales = L.w1_scales; g.zeros = L.w1_zeros; g.bias = L.b1;
    g.residual = nullptr; g.y = E.G; g.N = F; g.K = H; g.epi = Epi::BiasGelu;
    STEP(K_GEMM_FFN_UP, launch_gemm(g, ss));

    g.x = E.G; g.w = L.w2; g.scales = L.w2_scales; g.zeros = L.w2_zeros; g.bias = L.b2;
    g.residual = E.X1; g.y = E.A; g.N = H; g.K = F; g.epi = Epi::BiasResidual;
    STEP(K_GEMM_FFN_DOWN, launch_gemm(g, ss));
    STEP(K_LN2, launch_layer_norm(E.A, L.ln2_gamma, L.ln2_beta, c.ln_eps, H, n_dev, T, E.X, E.dt, ss));
  }
  const rlx_layer_weights& last = E.layers[c.layers - 1];
  if (c.output_kind == RLX_OUTPUT_POOLED) {
    // G (the last FFN-up output, consumed by now) holds the partial sums of long sequences
    float* pool_scratch = static_cast<float*>(E.G);
    const size_t pool_scratch_bytes = (size_t)T * F * (E.dt == DType::BF16 ? 2 : 4);
    if (E.deferred) {
      STEP(K_POOL, launch_pool_l2(E.X, H, E.cu, B, static_cast<float*>(output), E.dt, ss, E.S2,
                                  last.ln2_gamma, last.ln2_beta, c.ln_eps, c.quant != RLX_Q_NONE, S, pool_scratch,
                                  pool_scratch_bytes));
    } else {
      STEP(K_POOL, launch_pool_l2(E.X, H, E.cu, B, static_cast<float*>(output), E.dt, ss, nullptr, nullptr, nullptr,
                                  0.0f, false, S, pool_scratch, pool_scratch_bytes));
    }
  } else {
    const void* hid = E.X;
    if (E.deferred) {  // the hidden states are LN2's output: materialise it once
      STEP(K_LN2, launch_layer_norm(E.X, last.ln2_gamma, last.ln2_beta, c.ln_eps, H, n_dev, T, E.X1, E.dt, ss));
      hid = E.X1;
    }
    STEP(K_SCATTER, launch_scatter_hidden(hid, H, E.tok_dst, T, static_cast<float*>(output), E.dt, ss));
  }
#undef STEP
  return RLX_OK;
}

void destroy_graphs(rlx_encoder* e) {
  for (auto& g : e->graphs) (void)hipGraphExecDestroy(g.exec);
  e->graphs.clear();
  for (auto& g : e->prof_graphs)
    for (auto x : g.slot_exec) (void)hipGraphExecDestroy(x);
  e->prof_graphs.clear();
}

void clear_profile(rlx_encoder* e) {
  for (int c = 0; c < K_NUM_CLASSES; ++c) {
    e->prof_cnt[c] = 0;
    e->prof_ms[c] = 0.0;
  }
}

// Records the forward as a HIP graph on the capture stream; `slots` as in enqueue_forward.
rlx_status capture_forward(rlx_encoder* e, const void* input, const uint8_t* mask, int B, int S, void* output,
                           std::vector<KernelSlot>* slots, hipGraphExec_t* exec) {
  RLX_HIP(hipStreamBeginCapture(e->cap_stream, hipStreamCaptureModeThreadLocal), "hipStreamBeginCapture");
  rlx_status st = enqueue_forward(ctx_of(e, B, S), input, mask, B, S, output, e->cap_stream, slots);
  hipGraph_t graph = nullptr;
  hipError_t he = hipStreamEndCapture(e->cap_stream, &graph);
  if (st != RLX_OK) {
    if (graph) (void)hipGraphDestroy(graph);
    return st;
  }
  if (he != hipSuccess) return hip_fail(he, "hipStreamEndCapture");
  he = hipGraphInstantiate(exec, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  if (he != hipSuccess) return hip_fail(he, "hipGraphInstantiate");
  return RLX_OK;
}

// Profiled forward.  Per kernel of the forward, a graph of kProfReps
// back-to-back launches of that kernel alone (same arguments) is replayed
// between two events on the caller's stream; the mean is the kernel's time
// with only graph-replay gaps, like in the forward's own graph.  No kernel
// writes its own input, so repeats are idempotent.  A plain forward runs first
// (the token counts every kernel indexes with must be set for this mask) and
// again last, so the output is the forward's result.
rlx_status run_graph_forward(rlx_encoder* e, const void* input, const uint8_t* mask, int B, int S, void* output,
                             hipStream_t s);

rlx_status profiled_forward(rlx_encoder* e, const void* input, const uint8_t* mask, int B, int S, void* output,
                            hipStream_t s) {
  if (!e->prof_ev[0]) {
    RLX_HIP(hipEventCreate(&e->prof_ev[0]), "hipEventCreate");
    RLX_HIP(hipEventCreate(&e->prof_ev[1]), "hipEventCreate");
  }
  rlx_status st = run_graph_forward(e, input, mask, B, S, output, s);
  if (st != RLX_OK) return st;
  ProfGraph* hit = nullptr;
  for (auto& g : e->prof_graphs)
    if (g.g.B == B && g.g.S == S && g.g.input == input && g.g.mask == mask && g.g.output == output) hit = &g;
  if (!hit) {
    if (e->prof_graphs.size() >= kMaxGraphs) {
      RLX_HIP(hipEventSynchronize(e->done_ev), "hipEventSynchronize");
      for (auto x : e->prof_graphs.front().slot_exec) (void)hipGraphExecDestroy(x);
      e->prof_graphs.erase(e->prof_graphs.begin());
    }
    // record the launches of one forward (also a real forward on the capture stream)
    std::vector<KernelSlot> slots;
    RLX_HIP(hipStreamSynchronize(s), "hipStreamSynchronize");
    st = enqueue_forward(ctx_of(e, B, S), input, mask, B, S, output, e->cap_stream, &slots);
    if (st != RLX_OK) return st;
    RLX_HIP(hipStreamSynchronize(e->cap_stream), "hipStreamSynchronize");
    ProfGraph pg;
    pg.g = {B, S, input, mask, output, nullptr, 0};
    for (auto& sl : slots) {
      RLX_HIP(hipStreamBeginCapture(e->cap_stream, hipStreamCaptureModeThreadLocal), "hipStreamBeginCapture");
      hipError_t le = hipSuccess;
      for (int r = 0; r < kProfReps && le == hipSuccess; ++r) le = sl.launch(e->cap_stream);
      hipGraph_t graph = nullptr;
      hipError_t he = hipStreamEndCapture(e->cap_stream, &graph);
      if (le != hipSuccess || he != hipSuccess) {
        if (graph) (void)hipGraphDestroy(graph);
        return hip_fail(le != hipSuccess ? le : he, "profiling capture");
      }
      hipGraphExec_t x = nullptr;
      he = hipGraphInstantiate(&x, graph, nullptr, nullptr, 0);
      (void)hipGraphDestroy(graph);
      if (he != hipSuccess) return hip_fail(he, "hipGraphInstantiate");
      pg.slot_cls.push_back(sl.cls);
      pg.slot_exec.push_back(x);
    }
    e->prof_graphs.push_back(std::move(pg));
    hit = &e->prof_graphs.back();
  }
  for (size_t k = 0; k < hit->slot_exec.size(); ++k) {
    RLX_HIP(hipEventRecord(e->prof_ev[0], s), "hipEventRecord");
    RLX_HIP(hipGraphLaunch(hit->slot_exec[k], s), "hipGraphLaunch");
    RLX_HIP(hipEventRecord(e->prof_ev[1], s), "hipEventRecord");
    RLX_HIP(hipEventSynchronize(e->prof_ev[1]), "hipEventSynchronize");
    float t = 0.0f;
    RLX_HIP(hipEventElapsedTime(&t, e->prof_ev[0], e->prof_ev[1]), "hipEventElapsedTime");
    e->prof_cnt[hit->slot_cls[k]] += 1;
    e->prof_ms[hit->slot_cls[k]] += t / kProfReps;
  }
  return run_graph_forward(e, input, mask, B, S, output, s);
}

// The normal path: replay (recording on first use) the graph of this forward.
rlx_status run_graph_forward(rlx_encoder* e, const void* input, const uint8_t* mask, int B, int S, void* output,
                             hipStream_t s) {
  GraphEntry* hit = nullptr;
  for (auto& g : e->graphs)
    if (g.B == B && g.S == S && g.input == input && g.mask == mask && g.output == output) hit = &g;
  if (!hit) {
    if (e->graphs.size() >= kMaxGraphs) {
      auto lru = std::min_element(e->graphs.begin(), e->graphs.end(),
                                  [](const GraphEntry& a, const GraphEntry& b) { return a.last_use < b.last_use; });
      RLX_HIP(hipEventSynchronize(e->done_ev), "hipEventSynchronize");  // no replay of it is in flight
      (void)hipGraphExecDestroy(lru->exec);
      e->graphs.erase(lru);
    }
    hipGraphExec_t exec = nullptr;
    rlx_status st = capture_forward(e, input, mask, B, S, output, nullptr, &exec);
    if (st != RLX_OK) return st;
    e->graphs.push_back({B, S, input, mask, output, exec, 0});
    hit = &e->graphs.back();
  }
  hit->last_use = ++e->use_clock;
  RLX_HIP(hipGraphLaunch(hit->exec, s), "hipGraphLaunch");
  return RLX_OK;
}

// Deferred LayerNorm: folds each LayerNorm into the weights of the linear
// layer that reads it (LN1 into W1; LN2 of layer l-1 into Wqkv of layer l),
// once, on the capture stream, and waits for it.
rlx_status fold_layer_norms(rlx_encoder* e) {
  const rlx_encoder_config& c = e->cfg;
  const size_t H = c.hidden, F = c.ffn;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, 256); return o; };
  struct Offs { size_t wqkv, uq, vq, w1, u1, v1; };
  std::vector<Offs> offs(c.layers);
  // dense weights get gamma-scaled copies; quantised ones only the vectors
  // (their LN inputs travel gamma-scaled instead)
  const bool quant = c.quant != RLX_Q_NONE;
  for (int l = 0; l < c.layers; ++l) {
    if (l > 0) {
      if (!quant) offs[l].wqkv = take(3 * H * H * 2);
      offs[l].uq = take(3 * H * sizeof(float));
      offs[l].vq = take(3 * H * sizeof(float));
    }
    if (!quant) offs[l].w1 = take(F * H * 2);
    offs[l].u1 = take(F * sizeof(float));
    offs[l].v1 = take(F * sizeof(float));
  }
  hipError_t he = hipMalloc(&e->fold_mem, off);
  if (he != hipSuccess) {
    e->fold_mem = nullptr;
    return fail(RLX_ERR_OOM, "encoder_create: folded weights of %zu bytes: %s", off, hipGetErrorString(he));
  }
  uint8_t* base = static_cast<uint8_t*>(e->fold_mem);
  e->folded.assign(c.layers, rlx_encoder::Folded{});
  for (int l = 0; l < c.layers; ++l) {
    const rlx_layer_weights& L = e->layers[l];
    rlx_encoder::Folded& f = e->folded[l];
    const Quant q = to_quant(c.quant);
    if (l > 0) {
      const rlx_layer_weights& P = e->layers[l - 1];
      f.uq = reinterpret_cast<float*>(base + offs[l].uq);
      f.vq = reinterpret_cast<float*>(base + offs[l].vq);
      if (quant) {
        RLX_HIP(launch_fold_ln_quant(L.wqkv, q, L.wqkv_scales, L.wqkv_zeros, 3 * c.hidden, c.hidden, P.ln2_gamma,
                                     P.ln2_beta, L.bqkv, false, f.uq, f.vq, e->cap_stream),
                "encoder_create: fold LN2 into the QKV vectors");
      } else {
        f.wqkv = base + offs[l].wqkv;
        RLX_HIP(launch_fold_ln_weights(L.wqkv, 3 * c.hidden, c.hidden, P.ln2_gamma, P.ln2_beta, L.bqkv, f.wqkv,
                                       f.uq, f.vq, e->cap_stream),
                "encoder_create: fold LN2 into Wqkv");
      }
    }
    f.u1 = reinterpret_cast<float*>(base + offs[l].u1);
    f.v1 = reinterpret_cast<float*>(base + offs[l].v1);
    if (quant) {
      RLX_HIP(launch_fold_ln_quant(L.w1, q, L.w1_scales, L.w1_zeros, c.ffn, c.hidden, L.ln1_gamma, L.ln1_beta, L.b1,
                                   false, f.u1, f.v1, e->cap_stream),
              "encoder_create: fold LN1 into the FFN-up vectors");
    } else {
      f.w1 = base + offs[l].w1;
      RLX_HIP(launch_fold_ln_weights(L.w1, c.ffn, c.hidden, L.ln1_gamma, L.ln1_beta, L.b1, f.w1, f.u1, f.v1,
                                     e->cap_stream),
              "encoder_create: fold LN1 into W1");
    }
  }
  RLX_HIP(hipStreamSynchronize(e->cap_stream), "encoder_create: fold LayerNorms");
  return RLX_OK;
}

// Dequantisation prologue for a handle with quantised weights and the
// deferred LayerNorm: bf16 copies of every layer's matrices (refreshed by the
// first kernel of each large forward), with LN2 of layer l-1 folded into the
// QKV weights of layer l and LN1 into W1 as the dense path has them, their
// u / v vectors (over the same bf16(gamma * d) values), and the job table.
// RLX_DEQUANT_PROLOGUE_MIN_TOKENS overrides the size (B*S) from which a
// forward takes it; a negative value turns it off.  Measured on MiniLM-L6
// (per forward, dequantising GEMMs -> prologue): b1 int8 0.258 -> 0.197 ms,
// int4 0.356 -> 0.198; b4 0.281 -> 0.215, 0.375 -> 0.216; b32 0.331 -> 0.237,
// 0.437 -> 0.237.  The bf16 weights are converted once per forward instead of
// once per tile and wave that reads them, and the forward keeps the fused
// attention; so every size takes it.
constexpr int kDequantPrologueMinTokens = 0;

rlx_status setup_dequant_prologue(rlx_encoder* e) {
  const rlx_encoder_config& c = e->cfg;
  if (c.quant == RLX_Q_NONE || !e->deferred) return RLX_OK;
  int min_tokens = kDequantPrologueMinTokens;
  if (const char* env = std::getenv("RLX_DEQUANT_PROLOGUE_MIN_TOKENS")) min_tokens = std::atoi(env);
  if (min_tokens < 0) return RLX_OK;
  const size_t H = c.hidden, F = c.ffn, L = c.layers;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, 256); return o; };
  struct Offs { size_t wqkv, wo, w1, w2, uq, vq, u1, v1; };
  std::vector<Offs> offs(L);
  for (size_t l = 0; l < L; ++l) {
    offs[l].wqkv = take(3 * H * H * 2);
    offs[l].wo = take(H * H * 2);
    offs[l].w1 = take(F * H * 2);
    offs[l].w2 = take(H * F * 2);
    offs[l].uq = take(3 * H * sizeof(float));
    offs[l].vq = take(3 * H * sizeof(float));
    offs[l].u1 = take(F * sizeof(float));
    offs[l].v1 = take(F * sizeof(float));
  }
  const size_t jobs_off = take(4 * L * sizeof(DequantJob));
  RLX_HIP(hipMalloc(&e->dq_mem, off), "encoder_create: bf16 weight copies");
  uint8_t* base = static_cast<uint8_t*>(e->dq_mem);
  const Quant q = to_quant(c.quant);
  std::vector<DequantJob> jobs;
  e->dq_layers = e->layers;
  e->dq_folded.assign(L, rlx_encoder::Folded{});
  int max_elems = 0;
  auto job = [&](const void* w, const void* sc, const void* z, const float* gamma, void* out, int N, int K) {
    jobs.push_back(DequantJob{w, sc, z, gamma, out, N, K, q});
    max_elems = std::max(max_elems, N * K);
  };
  for (size_t l = 0; l < L; ++l) {
    const rlx_layer_weights& W = e->layers[l];
    rlx_layer_weights& D = e->dq_layers[l];
    rlx_encoder::Folded& f = e->dq_folded[l];
    void* wqkv = base + offs[l].wqkv;
    job(W.wqkv, W.wqkv_scales, W.wqkv_zeros, l > 0 ? e->layers[l - 1].ln2_gamma : nullptr, wqkv, 3 * H, H);
    job(W.wo, W.wo_scales, W.wo_zeros, nullptr, base + offs[l].wo, H, H);
    job(W.w1, W.w1_scales, W.w1_zeros, W.ln1_gamma, base + offs[l].w1, F, H);
    job(W.w2, W.w2_scales, W.w2_zeros, nullptr, base + offs[l].w2, H, F);
    D.wqkv = wqkv; D.wo = base + offs[l].wo; D.w1 = base + offs[l].w1; D.w2 = base + offs[l].w2;
    D.wqkv_scales = D.wqkv_zeros = D.wo_scales = D.wo_zeros = nullptr;
    D.w1_scales = D.w1_zeros = D.w2_scales = D.w2_zeros = nullptr;
    f.w1 = base + offs[l].w1;
    f.u1 = reinterpret_cast<float*>(base + offs[l].u1);
    f.v1 = reinterpret_cast<float*>(base + offs[l].v1);
    RLX_HIP(launch_fold_ln_quant(W.w1, q, W.w1_scales, W.w1_zeros, c.ffn, c.hidden, W.ln1_gamma, W.ln1_beta, W.b1, true,
                                 f.u1, f.v1, e->cap_stream),
            "encoder_create: fold LN1 (bf16 copies)");
    if (l > 0) {
      const rlx_layer_weights& P = e->layers[l - 1];
      f.wqkv = wqkv;
      f.uq = reinterpret_cast<float*>(base + offs[l].uq);
      f.vq = reinterpret_cast<float*>(base + offs[l].vq);
      RLX_HIP(launch_fold_ln_quant(W.wqkv, q, W.wqkv_scales, W.wqkv_zeros, 3 * c.hidden, c.hidden, P.ln2_gamma,
                                   P.ln2_beta, W.bqkv, true, f.uq, f.vq, e->cap_stream),
              "encoder_create: fold LN2 (bf16 copies)");
    }
  }
  RLX_HIP(hipMemcpyAsync(base + jobs_off, jobs.data(), jobs.size() * sizeof(DequantJob), hipMemcpyHostToDevice,
                         e->cap_stream),
          "encoder_create: dequantisation jobs");
  RLX_HIP(hipStreamSynchronize(e->cap_stream), "encoder_create: dequantisation setup");
  e->dq_jobs = reinterpret_cast<const DequantJob*>(base + jobs_off);
  e->dq_njobs = (int)jobs.size();
  e->dq_max_elems = max_elems;
  e->dq_cfg = c;
  e->dq_cfg.quant = RLX_Q_NONE;
  e->dq_min_tokens = min_tokens;
  return RLX_OK;
}

// Persistent forward: usable for a handle with dense bf16 weights, id input,
// pooled output and the hidden size its LDS plan is made for (the batch and
// sequence limits are checked per forward); selected when RLX_PIPELINE=1 is
// set in the environment.  Two blocks per CU.
rlx_status setup_pipeline(rlx_encoder* e) {
  const rlx_encoder_config& c = e->cfg;
  const char* env = std::getenv("RLX_PIPELINE");
  if (!env || env[0] != '1' || !e->deferred || c.quant != RLX_Q_NONE || c.input_kind != RLX_INPUT_IDS ||
      c.output_kind != RLX_OUTPUT_POOLED ||
      !pipe_supported(PipeShape{1, 16, c.hidden, c.ffn, c.heads, c.layers}) || c.layers > kPipeMaxLayers)
    return RLX_OK;
  int cus = 0;
  RLX_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, e->device), "hipDeviceGetAttribute");
  const int grid = 2 * cus;  // two blocks per CU
  if (grid <= 0) return RLX_OK;
  RLX_HIP(init_pipe_attributes(), "encoder_create: persistent-forward attributes");
  const size_t layer_bytes = align_up((size_t)c.layers * sizeof(PipeLayer), 256);
  const size_t bytes = layer_bytes + pipe_sync_bytes();
  hipError_t he = hipMalloc(&e->pipe_mem, bytes);
  if (he != hipSuccess) {
    e->pipe_mem = nullptr;
    return fail(RLX_ERR_OOM, "encoder_create: persistent-forward tables of %zu bytes: %s", bytes, hipGetErrorString(he));
  }
  uint8_t* base = static_cast<uint8_t*>(e->pipe_mem);
  e->pipe_layers = reinterpret_cast<PipeLayer*>(base);
  e->pipe_sync = reinterpret_cast<int*>(base + layer_bytes);
  std::vector<PipeLayer> host(c.layers);
  for (int l = 0; l < c.layers; ++l) {
    const rlx_layer_weights& L = e->layers[l];
    const rlx_encoder::Folded& f = e->folded[l];
    PipeLayer& P = host[l];
    P.wqkv = static_cast<const bf16_t*>(l > 0 ? f.wqkv : L.wqkv);
    P.bqkv = l > 0 ? f.vq : L.bqkv;
    P.uq = l > 0 ? f.uq : nullptr;
    P.wo = static_cast<const bf16_t*>(L.wo); P.bo = L.bo;
    P.res_g = l > 0 ? e->layers[l - 1].ln2_gamma : nullptr;
    P.res_b = l > 0 ? e->layers[l - 1].ln2_beta : nullptr;
    P.w1 = static_cast<const bf16_t*>(f.w1); P.v1 = f.v1; P.u1 = f.u1;
    P.w2 = static_cast<const bf16_t*>(L.w2); P.b2 = L.b2;
    P.ln1_g = L.ln1_gamma; P.ln1_b = L.ln1_beta;
  }
  RLX_HIP(hipMemcpyAsync(e->pipe_layers, host.data(), c.layers * sizeof(PipeLayer), hipMemcpyHostToDevice,
                         e->cap_stream), "encoder_create: persistent-forward layer table");
  RLX_HIP(hipMemsetAsync(e->pipe_sync, 0, pipe_sync_bytes(), e->cap_stream), "encoder_create: sync words");
  RLX_HIP(hipStreamSynchronize(e->cap_stream), "encoder_create: persistent-forward tables");
  e->pipe = true;
  e->pipe_grid = grid;
  return RLX_OK;
}

// ---------------------------------------------------------------------------
// Static scratch of the allocation-free forward
// ---------------------------------------------------------------------------
// One array per GPU, part of the library's code object: it exists from the
// first use of the library on that GPU until the process ends.  In host code
// `scratch` is only a host-side stand-in for the symbol; its device address is
// looked up once per device with hipGetSymbolAddress and used everywhere.
constexpr size_t kScratchBytes = (size_t)16 << 20;  // 16 MiB
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
uint8_t* g_scratch_ptr[kMaxScratchDevices] = {nullptr};

// Device address of this device's scratch (looked up on the first call with
// the device current).
rlx_status scratch_on_device(int dev, uint8_t** out) {
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(RLX_ERR_UNSUPPORTED, "encoder_forward_noalloc: device %d beyond the %d supported", dev,
                kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t he = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (he != hipSuccess || !ptr) return hip_fail(he, "encoder_forward_noalloc: hipGetSymbolAddress(scratch)");
    g_scratch_ptr[dev] = static_cast<uint8_t*>(ptr);
  }
  *out = g_scratch_ptr[dev];
  return RLX_OK;
}

}  // namespace

bool rlx::g_log_launches = false;

void rlx::log_launch(const char* kernel, dim3 grid, dim3 block, size_t lds, const char* fmt, ...) {
  char detail[256];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(detail, sizeof(detail), fmt, ap);
  va_end(ap);
  std::fprintf(stderr, "[rlx] %s %s grid=(%u,%u,%u) block=%u lds=%zu\n", kernel, detail, grid.x, grid.y, grid.z,
               block.x, lds);
}

namespace {
// Every entry point re-reads RLX_LOG, so a caller can switch the log on or off
// between calls.
void log_refresh() {
  const char* v = std::getenv("RLX_LOG");
  g_log_launches = v && v[0] == '1';
}
}  // namespace

extern "C" {

const char* rlx_last_error(void) { return g_last_error.c_str(); }

const char* rlx_version(void) { return "rlx-mi355x 0.1.0 (gfx950)"; }

rlx_status rlx_masked_attention(const void* q, const void* k, const void* v, int64_t qkv_row_stride, void* out,
                                int64_t out_row_stride, int B, int S, int num_heads, int head_dim, rlx_dtype dt,
                                rlx_mask_kind kind, const uint8_t* key_mask, int window, float scale,
                                void* stream) {
  log_refresh();
  rlx_status st = check_attention_args(q, k, v, qkv_row_stride, out, out_row_stride, B, S, num_heads, head_dim, dt,
                                       kind, key_mask, window, scale);
  if (st != RLX_OK) return st;
  if (B == 0 || S == 0) return ok();
  AttnParams a{};
  a.q = q; a.k = k; a.v = v; a.ld_qkv = qkv_row_stride;
  a.out = out; a.ld_out = out_row_stride;
  a.B = B; a.S = S; a.heads = num_heads; a.kind = (int)kind; a.key_mask = key_mask; a.window = window;
  a.scale = scale; a.cu_seqlens = nullptr;
  a.dtype = dt == RLX_BF16 ? DType::BF16 : DType::F32;
  RLX_HIP(launch_attention(a, static_cast<hipStream_t>(stream)), "attention launch");
  return ok();
}

rlx_status rlx_dequant_matmul(const void* x, rlx_dtype x_dt, int M, int K, const void* w, rlx_quant scheme,
                              const void* scales, const void* zeros, int group_size, int N, const float* bias,
                              const void* residual, rlx_epilogue epi, void* y, rlx_dtype y_dt, void* stream) {
  log_refresh();
  if (M < 0 || N <= 0 || K <= 0)
    return fail(RLX_ERR_INVALID_ARG, "dequant_matmul: M=%d must be >= 0, N=%d and K=%d positive", M, N, K);
  if (!x || !y) return fail(RLX_ERR_INVALID_ARG, "dequant_matmul: x and y must be non-null");
  if (epi < RLX_EPI_NONE || epi > RLX_EPI_BIAS_RESIDUAL)
    return fail(RLX_ERR_INVALID_ARG, "dequant_matmul: unknown epilogue %d", (int)epi);
  if (epi != RLX_EPI_NONE && !bias) return fail(RLX_ERR_INVALID_ARG, "dequant_matmul: epilogue needs a bias");
  if (epi == RLX_EPI_BIAS_RESIDUAL && !residual)
    return fail(RLX_ERR_INVALID_ARG, "dequant_matmul: residual epilogue needs a residual");
  if (x_dt != RLX_BF16 && x_dt != RLX_F32)
    return fail(RLX_ERR_UNSUPPORTED, "dequant_matmul: activation dtype %s not supported (bf16, f32)",
                dtype_name(x_dt));
  if (y_dt != x_dt && !(x_dt == RLX_BF16 && y_dt == RLX_F32))
    return fail(RLX_ERR_UNSUPPORTED, "dequant_matmul: output dtype %s with %s activations not supported "
                "(bf16 -> bf16 or f32, f32 -> f32)", dtype_name(y_dt), dtype_name(x_dt));
  rlx_status st = check_quant_weights("dequant_matmul", scheme, w, scales, zeros, group_size, N, K);
  if (st != RLX_OK) return st;
  if (scheme != RLX_Q_NONE && x_dt != RLX_BF16)
    return fail(RLX_ERR_UNSUPPORTED, "dequant_matmul: quantised weights need bf16 activations");
  if (!aligned16(x) || !aligned16(y) || (residual && !aligned16(residual)) || (bias && !aligned16(bias)))
    return fail(RLX_ERR_UNSUPPORTED, "dequant_matmul: x, y, bias and residual must be 16-byte aligned");
  if (M == 0) return ok();
  GemmParams g{};
  g.x = x; g.w = w; g.scales = scales; g.zeros = zeros; g.bias = bias; g.residual = residual; g.y = y;
  g.M = M; g.N = N; g.K = K; g.m_dev = nullptr;
  g.dtype = x_dt == RLX_BF16 ? DType::BF16 : DType::F32;
  g.quant = to_quant(scheme);
  g.epi = static_cast<Epi>(epi);
  g.y_f32 = x_dt == RLX_BF16 && y_dt == RLX_F32;
  RLX_HIP(launch_gemm(g, static_cast<hipStream_t>(stream)), "gemm launch");
  return ok();
}

rlx_status rlx_scaled_matmul(const void* x, const uint8_t* x_scales, rlx_mx_format fx, const void* w,
                             const uint8_t* w_scales, rlx_mx_format fw, int M, int N, int K, float* y,
                             void* stream) {
  log_refresh();
  if (M < 0 || N <= 0 || K <= 0)
    return fail(RLX_ERR_INVALID_ARG, "scaled_matmul: M=%d must be >= 0, N=%d and K=%d positive", M, N, K);
  if (fx < RLX_MX_E4M3 || fx > RLX_MX_E2M1 || fw < RLX_MX_E4M3 || fw > RLX_MX_E2M1)
    return fail(RLX_ERR_INVALID_ARG, "scaled_matmul: unknown element format (%d, %d)", (int)fx, (int)fw);
  if (!w || !w_scales || (M > 0 && (!x || !x_scales || !y)))
    return fail(RLX_ERR_INVALID_ARG, "scaled_matmul: x, x_scales, w, w_scales and y must be non-null");
  if (!mx_gemm_supported(M, N, K))
    return fail(RLX_ERR_UNSUPPORTED, "scaled_matmul: N=%d and K=%d must be multiples of 128", N, K);
  if (!aligned16(x) || !aligned16(w) || !aligned16(y) || (reinterpret_cast<uintptr_t>(x_scales) & 3) ||
      (reinterpret_cast<uintptr_t>(w_scales) & 3))
    return fail(RLX_ERR_UNSUPPORTED, "scaled_matmul: x, w, y must be 16-byte and the scales 4-byte aligned");
  if (M == 0) return ok();  // (x, x_scales and y may then be null)
  MxGemmParams p{};
  p.x = x; p.x_scales = x_scales; p.fx = (int)fx;
  p.w = w; p.w_scales = w_scales; p.fw = (int)fw;
  p.y = y; p.M = M; p.N = N; p.K = K;
  RLX_HIP(launch_mx_gemm(p, static_cast<hipStream_t>(stream)), "scaled matmul launch");
  return ok();
}

rlx_status rlx_dequant_unpack(const void* w, rlx_quant scheme, const void* scales, const void* zeros, int group_size,
                              int N, int K, float* w_out, void* stream) {
  log_refresh();
  if (N <= 0 || K <= 0) return fail(RLX_ERR_INVALID_ARG, "dequant_unpack: N=%d and K=%d must be positive", N, K);
  if (!w_out) return fail(RLX_ERR_INVALID_ARG, "dequant_unpack: w_out must be non-null");
  if (scheme == RLX_Q_NONE) return fail(RLX_ERR_INVALID_ARG, "dequant_unpack: scheme must be a quantised one");
  rlx_status st = check_quant_weights("dequant_unpack", scheme, w, scales, zeros, group_size, N, K);
  if (st != RLX_OK) return st;
  RLX_HIP(launch_dequant_unpack(w, to_quant(scheme), scales, zeros, N, K, w_out, static_cast<hipStream_t>(stream)),
          "dequant unpack launch");
  return ok();
}

rlx_status rlx_gguf_repack(const void* blocks, rlx_gguf_type type, int N, int K, void* codes, void* scales,
                           void* zeros, rlx_quant* scheme, void* stream) {
  log_refresh();
  if (type != RLX_GGUF_Q4_0 && type != RLX_GGUF_Q4_1 && type != RLX_GGUF_Q8_0 && type != RLX_GGUF_Q4_K &&
      type != RLX_GGUF_Q6_K)
    return fail(RLX_ERR_UNSUPPORTED,
                "gguf_repack: tensor type %d not supported (Q4_0 2, Q4_1 3, Q8_0 8, Q4_K 12, Q6_K 14)", (int)type);
  if (N < 0 || K <= 0) return fail(RLX_ERR_INVALID_ARG, "gguf_repack: N=%d must be >= 0 and K=%d positive", N, K);
  const bool kquant = type == RLX_GGUF_Q4_K || type == RLX_GGUF_Q6_K;
  if (K % (kquant ? 256 : 64))
    return fail(RLX_ERR_UNSUPPORTED, "gguf_repack: K=%d must be a multiple of %d", K, kquant ? 256 : 64);
  const bool four = type != RLX_GGUF_Q8_0 && type != RLX_GGUF_Q6_K;  // a zeros / mins array
  if (N > 0 && (!blocks || !codes || !scales || (four && !zeros)))
    return fail(RLX_ERR_INVALID_ARG, "gguf_repack: blocks, codes, scales%s must be non-null", four ? " and zeros" : "");
  if ((reinterpret_cast<uintptr_t>(blocks) & 1) || !aligned16(codes) || (reinterpret_cast<uintptr_t>(scales) & 1) ||
      (four && (reinterpret_cast<uintptr_t>(zeros) & 1)))
    return fail(RLX_ERR_UNSUPPORTED, "gguf_repack: blocks, scales and zeros must be 2-byte, codes 16-byte aligned");
  if (scheme)
    *scheme = type == RLX_GGUF_Q4_0                            ? RLX_Q_INT4_GROUP_ZP
              : (type == RLX_GGUF_Q4_1 || type == RLX_GGUF_Q4_K) ? RLX_Q_INT4_GROUP_MIN
              : type == RLX_GGUF_Q6_K                          ? RLX_Q_INT8_GROUP16
                                                               : RLX_Q_INT8_GROUP;
  RLX_HIP(launch_gguf_repack(blocks, (int)type, N, K, codes, scales, zeros, static_cast<hipStream_t>(stream)),
          "gguf repack launch");
  return ok();
}

rlx_status rlx_encoder_create(const rlx_encoder_config* cfg, const rlx_encoder_weights* w, rlx_encoder** out) {
  log_refresh();
  if (!cfg || !w || !out) return fail(RLX_ERR_INVALID_ARG, "encoder_create: cfg, weights and out must be non-null");
  *out = nullptr;
  rlx_status st = check_config(cfg);
  if (st != RLX_OK) return st;
  st = check_weights(cfg, w);
  if (st != RLX_OK) return st;

  rlx_encoder* e = new rlx_encoder();
  e->cfg = *cfg;
  e->w = *w;
  e->layers.assign(w->layers, w->layers + cfg->layers);
  e->w.layers = e->layers.data();
  e->dt = cfg->dtype == RLX_BF16 ? DType::BF16 : DType::F32;
  hipError_t he = hipGetDevice(&e->device);
  if (he == hipSuccess) he = init_kernel_attributes();  // outside any graph capture
  if (he != hipSuccess) {
    delete e;
    return hip_fail(he, "encoder_create: device setup");
  }

  // Workspace plan: token maps, then six activation buffers for T_max tokens.
  const size_t es = e->dt == DType::BF16 ? 2 : 4;
  // Quantised weights: the deferred LayerNorm stores LN inputs gamma-scaled,
  // so the final hidden states would need their own normalisation kernel;
  // pooled outputs only.
  e->deferred = gemm_deferred_ln_supported(e->dt, to_quant(cfg->quant), cfg->hidden) &&
                (cfg->quant == RLX_Q_NONE || cfg->output_kind == RLX_OUTPUT_POOLED);
  const WsPlan plan = plan_workspace(cfg->max_batch, cfg->max_seq, cfg->hidden, cfg->ffn, es, e->deferred);
  he = hipMalloc(&e->ws, plan.bytes);
  if (he != hipSuccess) {
    delete e;
    return fail(RLX_ERR_OOM, "encoder_create: workspace of %zu bytes: %s", plan.bytes, hipGetErrorString(he));
  }
  {
    FwdCtx view{};
    view.deferred = e->deferred;
    bind_workspace(view, static_cast<uint8_t*>(e->ws), plan);
    e->cu = view.cu; e->tok_src = view.tok_src; e->tok_dst = view.tok_dst; e->order = view.order;
    e->rank_rows = view.rank_rows;
    e->X = view.X; e->X1 = view.X1; e->A = view.A; e->CTX = view.CTX; e->QKV = view.QKV; e->G = view.G;
    e->S1 = view.S1; e->S2 = view.S2;
  }
  he = hipStreamCreateWithFlags(&e->cap_stream, hipStreamNonBlocking);
  if (he == hipSuccess) he = hipEventCreateWithFlags(&e->done_ev, hipEventDisableTiming);
  if (he != hipSuccess) {
    rlx_encoder_destroy(e);
    return hip_fail(he, "encoder_create: stream and event");
  }
  if (e->deferred) {
    st = fold_layer_norms(e);
    if (st == RLX_OK) st = setup_dequant_prologue(e);
    if (st == RLX_OK) st = setup_pipeline(e);
    if (st != RLX_OK) {
      rlx_encoder_destroy(e);
      return st;
    }
  }
  *out = e;
  return ok();
}

rlx_status rlx_encoder_forward(rlx_encoder* e, const void* input, const uint8_t* attention_mask, int B, int S,
                               void* output, void* stream) {
  log_refresh();
  if (!e) return fail(RLX_ERR_INVALID_ARG, "encoder_forward: null handle");
  if (!input || !attention_mask || !output)
    return fail(RLX_ERR_INVALID_ARG, "encoder_forward: input, attention_mask and output must be non-null");
  if (B < 1 || S < 1) return fail(RLX_ERR_INVALID_ARG, "encoder_forward: B=%d and S=%d must be >= 1", B, S);
  if (B > e->cfg.max_batch || S > e->cfg.max_seq)
    return fail(RLX_ERR_UNSUPPORTED, "encoder_forward: B=%d, S=%d exceed the planned max_batch=%d, max_seq=%d", B,
                S, e->cfg.max_batch, e->cfg.max_seq);
  int dev = -1;
  RLX_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (dev != e->device)
    return fail(RLX_ERR_INVALID_ARG, "encoder_forward: current device %d differs from the handle's device %d", dev,
                e->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (g_log_launches) {
    const FwdCtx c = ctx_of(e, B, S);
    std::fprintf(stderr, "[rlx] encoder_forward B=%d S=%d layers=%d %s%s%s%s\n", B, S, e->cfg.layers,
                 e->dt == DType::BF16 ? "bf16" : "f32", c.dq_njobs ? ", dequantisation prologue" : "",
                 c.pipe_grid > 0 ? ", persistent" : "",
                 e->profiling ? ", profiled" : e->cfg.use_graph ? ", graph (launches below only when recorded)" : "");
  }
  rlx_status st;
  if (e->profiling)
    st = profiled_forward(e, input, attention_mask, B, S, output, s);
  else if (!e->cfg.use_graph)
    st = enqueue_forward(ctx_of(e, B, S), input, attention_mask, B, S, output, s, nullptr);
  else
    st = run_graph_forward(e, input, attention_mask, B, S, output, s);
  if (st != RLX_OK) return st;
  RLX_HIP(hipEventRecord(e->done_ev, s), "hipEventRecord");
  e->last_B = B;
  e->last_S = S;
  return ok();
}

rlx_status rlx_encoder_forward_noalloc(const rlx_encoder_config* cfg, const rlx_encoder_weights* w,
                                       const void* input, const uint8_t* attention_mask, int B, int S, void* output,
                                       void* stream) {
  log_refresh();
  if (!cfg || !w) return fail(RLX_ERR_INVALID_ARG, "encoder_forward_noalloc: cfg and weights must be non-null");
  rlx_status st = check_config(cfg);
  if (st != RLX_OK) return st;
  st = check_weights(cfg, w);
  if (st != RLX_OK) return st;
  if (!input || !attention_mask || !output)
    return fail(RLX_ERR_INVALID_ARG, "encoder_forward_noalloc: input, attention_mask and output must be non-null");
  if (B < 1 || S < 1) return fail(RLX_ERR_INVALID_ARG, "encoder_forward_noalloc: B=%d and S=%d must be >= 1", B, S);
  if (S > 512) return fail(RLX_ERR_UNSUPPORTED, "encoder_forward_noalloc: S=%d exceeds 512", S);
  if (cfg->input_kind == RLX_INPUT_IDS && S > cfg->max_pos)
    return fail(RLX_ERR_UNSUPPORTED, "encoder_forward_noalloc: S=%d exceeds max_pos=%d", S, cfg->max_pos);
  const DType dt = cfg->dtype == RLX_BF16 ? DType::BF16 : DType::F32;
  const size_t es = dt == DType::BF16 ? 2 : 4;
  // the plain-LayerNorm kernel sequence: no LayerNorm-folded weights to allocate
  const WsPlan plan = plan_workspace((size_t)B, (size_t)S, cfg->hidden, cfg->ffn, es, false);
  if (plan.bytes > kScratchBytes)
    return fail(RLX_ERR_UNSUPPORTED,
                "encoder_forward_noalloc: B=%d x S=%d needs %zu bytes of workspace, the static scratch holds %zu",
                B, S, plan.bytes, kScratchBytes);
  int dev = -1;
  RLX_HIP(hipGetDevice(&dev), "hipGetDevice");
  uint8_t* base = nullptr;
  st = scratch_on_device(dev, &base);
  if (st != RLX_OK) return st;
  RLX_HIP(init_kernel_attributes(), "encoder_forward_noalloc: kernel attributes");
  FwdCtx c{};
  c.cfg = cfg;
  c.w = w;
  c.layers = w->layers;
  c.dt = dt;
  c.deferred = false;
  c.folded = nullptr;
  bind_workspace(c, base, plan);
  st = enqueue_forward(c, input, attention_mask, B, S, output, static_cast<hipStream_t>(stream), nullptr);
  return st == RLX_OK ? ok() : st;
}

void rlx_encoder_destroy(rlx_encoder* e) {
  if (!e) return;
  // the last forward enqueued through the handle, and the handle's own stream
  if (e->done_ev) (void)hipEventSynchronize(e->done_ev);
  if (e->cap_stream) (void)hipStreamSynchronize(e->cap_stream);
  destroy_graphs(e);
  for (auto ev : e->prof_ev)
    if (ev) (void)hipEventDestroy(ev);
  if (e->done_ev) (void)hipEventDestroy(e->done_ev);
  if (e->cap_stream) (void)hipStreamDestroy(e->cap_stream);
  if (e->ws) (void)hipFree(e->ws);
  if (e->fold_mem) (void)hipFree(e->fold_mem);
  if (e->dq_mem) (void)hipFree(e->dq_mem);
  if (e->pipe_mem) (void)hipFree(e->pipe_mem);
  delete e;
}

rlx_status rlx_encoder_check(rlx_encoder* e) {
  if (!e) return fail(RLX_ERR_INVALID_ARG, "encoder_check: null handle");
  RLX_HIP(hipEventSynchronize(e->done_ev), "hipEventSynchronize");
  if (!e->pipe) return ok();
  // the sticky error word of each XCD (word 3 of its sync block)
  int err[8] = {0};
  for (int x = 0; x < 8; ++x)
    RLX_HIP(hipMemcpyAsync(&err[x], e->pipe_sync + (size_t)x * kPipeSyncStride + 3, sizeof(int),
                           hipMemcpyDeviceToHost, e->cap_stream), "encoder_check: read");
  RLX_HIP(hipStreamSynchronize(e->cap_stream), "encoder_check: read");
  int all = 0;
  for (int x = 0; x < 8; ++x) {
    if (err[x])
      RLX_HIP(hipMemsetAsync(e->pipe_sync + (size_t)x * kPipeSyncStride + 3, 0, sizeof(int), e->cap_stream),
              "encoder_check: clear");
    all |= err[x];
  }
  RLX_HIP(hipStreamSynchronize(e->cap_stream), "encoder_check: clear");
  if (all)
    return fail(RLX_ERR_HIP, "encoder_check: a wait of the persistent forward gave up; its outputs are not valid");
  return ok();
}

int rlx_encoder_uses_persistent_forward(const rlx_encoder* e) { return e && e->pipe ? 1 : 0; }

rlx_status rlx_mask_compaction(const uint8_t* attention_mask, int B, int S, int32_t* cu, int32_t* tok_src,
                               int32_t* tok_dst, int32_t* order, void* stream) {
  log_refresh();
  if (!attention_mask || !cu || !tok_src || !tok_dst)
    return fail(RLX_ERR_INVALID_ARG, "mask_compaction: attention_mask, cu, tok_src and tok_dst must be non-null");
  if (B < 1 || S < 1) return fail(RLX_ERR_INVALID_ARG, "mask_compaction: B=%d and S=%d must be >= 1", B, S);
  if (B > 8192 || S > 512)
    return fail(RLX_ERR_UNSUPPORTED, "mask_compaction: B=%d, S=%d beyond B <= 8192, S <= 512", B, S);
  if (order && B > kMaxOrderedBatch)
    return fail(RLX_ERR_UNSUPPORTED, "mask_compaction: the order is computed for B <= %d, not %d", kMaxOrderedBatch, B);
  RLX_HIP(launch_mask_scan(attention_mask, B, S, cu, tok_src, tok_dst, order, static_cast<hipStream_t>(stream)),
          "mask compaction launch");
  return ok();
}

rlx_status rlx_encoder_token_maps(const rlx_encoder* e, int B, int S, int32_t* cu, int32_t* tok_src,
                                  int32_t* tok_dst, int32_t* order, void* stream) {
  log_refresh();
  if (!e) return fail(RLX_ERR_INVALID_ARG, "encoder_token_maps: null handle");
  if (!cu || !tok_src || !tok_dst)
    return fail(RLX_ERR_INVALID_ARG, "encoder_token_maps: cu, tok_src and tok_dst must be non-null");
  if (e->pipe) return fail(RLX_ERR_UNSUPPORTED, "encoder_token_maps: the persistent forward keeps no maps");
  if (e->last_B < 1 || B != e->last_B || S != e->last_S)
    return fail(RLX_ERR_INVALID_ARG, "encoder_token_maps: B=%d, S=%d differ from the most recent forward's %d, %d", B,
                S, e->last_B, e->last_S);
  if (order && B > kMaxOrderedBatch)
    return fail(RLX_ERR_UNSUPPORTED, "encoder_token_maps: the order is kept for B <= %d, not %d", kMaxOrderedBatch, B);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t n = (size_t)B * S * sizeof(int32_t);
  RLX_HIP(hipMemcpyAsync(cu, e->cu, (size_t)(B + 1) * sizeof(int32_t), hipMemcpyDeviceToDevice, s), "copy cu");
  RLX_HIP(hipMemcpyAsync(tok_src, e->tok_src, n, hipMemcpyDeviceToDevice, s), "copy tok_src");
  RLX_HIP(hipMemcpyAsync(tok_dst, e->tok_dst, n, hipMemcpyDeviceToDevice, s), "copy tok_dst");
  if (order)
    RLX_HIP(hipMemcpyAsync(order, e->order, (size_t)B * sizeof(int32_t), hipMemcpyDeviceToDevice, s), "copy order");
  return ok();
}

rlx_status rlx_encoder_set_profiling(rlx_encoder* e, int enable) {
  if (!e) return fail(RLX_ERR_INVALID_ARG, "encoder_set_profiling: null handle");
  e->profiling = enable != 0;
  clear_profile(e);
  return ok();
}

rlx_status rlx_encoder_profile_read(rlx_encoder* e, int max_entries, const char** names, int* launches,
                                    double* total_ms, int* n_entries) {
  if (!e || !n_entries) return fail(RLX_ERR_INVALID_ARG, "encoder_profile_read: null handle or n_entries");
  if (max_entries < 0 || (max_entries > 0 && (!names || !launches || !total_ms)))
    return fail(RLX_ERR_INVALID_ARG, "encoder_profile_read: output arrays required for max_entries > 0");
  const int* cnt = e->prof_cnt;
  const double* ms = e->prof_ms;
  int n = 0;
  for (int c = 0; c < K_NUM_CLASSES; ++c) {
    if (!cnt[c]) continue;
    if (n < max_entries) {
      names[n] = kClassNames[c];
      launches[n] = cnt[c];
      total_ms[n] = ms[c];
    }
    ++n;
  }
  *n_entries = n;
  clear_profile(e);
  return ok();
}

}  // extern "C"
