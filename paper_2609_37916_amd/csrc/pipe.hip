// Persistent encoder forward for gfx950: the whole bf16 forward of the
// MiniLM-shaped encoder (embedding gather + LayerNorm, every post-LN layer,
// masked mean-pool + L2 normalisation; Section VIII-B's inference workload) in
// one launch, for sequences of at most 128 tokens.
//
// Why one launch: at batch 32 x 128 the forward holds ~20 us of matrix work at
// peak, split over 26 dependent kernels when launched one by one; each of
// those pays a launch gap, a first-load round trip (~1.3 us) and a drained
// epilogue, which together cost more than the work.  Here the same tiles run
// back to back inside resident blocks, each tile's weights are requested
// before its inputs are ready, and a tile starts as soon as the tiles it reads
// are done.
//
// Dependencies stay inside one XCD.  Sequences never exchange data, so the
// batch is cut into eight contiguous runs of sequences with about equal token
// counts, one per XCD, and the blocks running on an XCD (HW_REG_XCC_ID) work
// only on that XCD's rows.  All producers and consumers of a row then share
// one L2, so a hand-off needs no L2 write-back: the producer's stores are
// complete in L2 once its vector-memory counter drains (s_waitcnt vmcnt(0)),
// after which it bumps a completion counter with a device-scope atomic (also
// performed in that L2); the consumer polls the counter with device-scope
// loads (which miss its L1), then invalidates its L1 before reading.
//
// Work items of an XCD, in queue order (every item depends only on items
// earlier in the queue, so the blocks that took them are running and the
// waits always end; each wait is also bounded):
//   E   embedding of 16 rows
//   per layer l:
//     A  (sequence, head): QKV projection + attention (qkv_attention_block),
//        after the sequence's rows of the previous layer (or E) are done
//     O  (64-row tile, 64 columns): output projection + bias + residual, and
//        the partial LayerNorm statistics of its output (LN1 deferred), after
//        every head of every sequence in the row tile
//     U  (64-row tile, 128 columns): FFN-up on the LayerNorm-folded W1 + bias +
//        erf-GELU, after the row tile's O tiles
//     D  (64-row tile, 64 columns): FFN-down + bias + LN1(residual) and the
//        statistics of its output (LN2 deferred), after the row tile's U tiles
//   P   per sequence: LN2 of the last layer, masked mean, L2 normalisation
// Each block takes the next item from its XCD's queue (an atomic counter),
// requests the item's weights, waits for the item's inputs, computes, and
// bumps the item's completion counter.  The counters start at zero: a small
// clear kernel runs before every launch (kernel boundaries make its stores
// visible to every XCD).  Nothing assumes which XCD a block runs on, or that
// all blocks are resident at once.
#include <math.h>

#include "common.hpp"
#include "gemm_tile.hpp"
#include "kernels.hpp"
#include "qkv_attention.hpp"

namespace rlx {
namespace {

constexpr int kPThreads = 256;
constexpr int kPStateBytes = 2048;  // block state at the start of the LDS
constexpr int kPItemBytes = kPipeLdsBytes - kPStateBytes;
constexpr int kSpinLimit = 1 << 20;  // polls before a wait gives up (~0.5 s)
constexpr int kRowTile = 64;
constexpr int kUpCols = 128;  // FFN-up column tile; the N = H products use 64
constexpr int kEmbRows = 16;  // rows per embedding item (4 per wave)
constexpr int kPoolBatch = 16;  // rows per wave in flight when pooling

// Per-XCD sync words (ints; each XCD's block is kPipeSyncStride ints).
constexpr int kQueue = 0, kAbort = 2, kErr = 3, kCntE = 32, kCntP = 33, kCntBase = 64;
__host__ __device__ constexpr int cnt_a(int l, int s) { return kCntBase + l * kPipeMaxBatch + s; }
__host__ __device__ constexpr int cnt_tile(int which, int L, int l, int rt) {  // which: 0 O, 1 U, 2 D
  return kCntBase + L * kPipeMaxBatch + (which * L + l) * kPipeMaxRowTiles + rt;
}

struct PipeState {
  int cu[kPipeMaxBatch + 1];  // row offsets of the sequences (exclusive prefix of the token counts)
  int seq0, seq1;             // this XCD's sequences
  int row0, row1;             // and rows
  int nrt, total;             // row tiles, items
  int item;                   // broadcast slot
};
static_assert(sizeof(PipeState) <= kPStateBytes, "state");

__device__ __forceinline__ int xcc_id() {
  return (int)(__builtin_amdgcn_s_getreg((20) | (0 << 6) | ((16 - 1) << 11)) & 0xf);  // HW_REG_XCC_ID
}

// Values every lane of the block holds alike, made scalar: branches and loop
// bounds on them compile to scalar branches.  (A loop whose exit the compiler
// takes to be per-lane is restructured with lane masks, and a barrier inside
// it can then run a different number of times in different waves.)
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
template <typename T>
__device__ __forceinline__ T* uni_ptr(T* p) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a), hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  return reinterpret_cast<T*>(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ int ld_acquire_cnt(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Thread 0: wait until sy[idx] >= target, or give up (sets the XCD's abort
// word and the sticky error word); returns at once once the XCD has aborted.
__device__ __forceinline__ void wait_count(int* sy, int idx, int target) {
  for (int n = 0; n < kSpinLimit; ++n) {
    if (ld_acquire_cnt(sy + idx) >= target) return;
    if ((n & 63) == 63 && ld_acquire_cnt(sy + kAbort) != 0) return;
    __builtin_amdgcn_s_sleep(1);
  }
  __hip_atomic_store(sy + kAbort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_fetch_or(sy + kErr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Every thread: after thread 0's waits, make the producers' rows visible.
__device__ __forceinline__ void finish_wait() {
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");  // invalidates this CU's L1
}

// Sequence (of this XCD) holding global row g: the largest b in [seq0, seq1)
// with cu[b] <= g (empty sequences share their offset with the next one).
__device__ __forceinline__ int seq_of_row(const PipeState& S, int g) {
  int lo = S.seq0, hi = S.seq1 - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (S.cu[mid] <= g) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// An item's inputs: counters sy[first .. last] must each reach `target`
// (contiguous: the heads of consecutive sequences, or the tiles of
// consecutive row tiles).  Called by every thread; thread 0 polls.
struct DepWait {
  int* sy;
  int first, last, target;
  __device__ __forceinline__ void operator()() const {
    int* const s = uni_ptr(sy);
    const int lo = uni(first), hi = uni(last), t = uni(target);
    if (threadIdx.x == 0)
      for (int i = lo; i <= hi; ++i) wait_count(s, i, t);
    finish_wait();
  }
};

// ---------------------------------------------------------------------------
// GEMM tile item: y[m0 .. m0+BM, n0 .. n0+BN] of the dense bf16 product with
// the fused epilogue (gemm_tile.hpp), rows at or past p.M clamped / skipped.
// 256 threads, 4 waves in a 2 x 2 grid; 64-k stages by LDS DMA in a ring of
// STAGES.  The weight rows of the first stages are requested before
// wait_inputs(), the activations, residual and statistics after it.
// ---------------------------------------------------------------------------
template <int BM, int BN, int STAGES>
constexpr int gemm_item_ring_bytes() { return STAGES * (BM + BN) * kRowBytes; }

template <int BM, int BN, int STAGES, Epi E, int LN, typename Wait>
__device__ __forceinline__ void gemm_item(const GemmParams& p, uint8_t* smem, int m0, int n0, Wait&& wait_inputs) {
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int kStage = (BM + BN) * kRowBytes;
  constexpr int XI = BM / 8, WI = BN / 8;  // 1 KB DMA blocks of a stage: activations, then weights
  constexpr int LPS = (XI + WI) / 4;        // DMA instructions per wave per stage
  constexpr int XL = XI / 4;                // of which activations (the first XL)
  static_assert(XI % 4 == 0 && WI % 4 == 0 && STAGES >= 2, "tile");
  static_assert((STAGES - 2) * LPS < 64, "vmcnt range");
  uint8_t* epi = smem + STAGES * kStage;
  const int M = uni(p.M);
  m0 = uni(m0);
  n0 = uni(n0);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, half = lane >> 5;
  const int K = uni(p.K);
  const int KT = K / 64;
  const size_t pitch = (size_t)K * 2;
  // activations row-major, or head-major ([K/32][x_head_rows][32]) from the
  // fused attention: a 64-k stage spans two heads, logical chunk c sits in
  // head c / 4 at dims (c % 4) * 8
  const bool head_major = p.x_head_rows > 0;
  const size_t x_stage = head_major ? (size_t)2 * p.x_head_rows * 64 : kRowBytes;
  const uint8_t* src[LPS];
#pragma unroll
  for (int i = 0; i < LPS; ++i) {
    const int g = wave + i * 4;
    if (i < XL) {
      const int row = 8 * g + (lane >> 3);
      const int c = swz(row, lane & 7);
      const int m = min(m0 + row, M - 1);
      src[i] = head_major ? reinterpret_cast<const uint8_t*>(p.x) + ((size_t)(c >> 2) * p.x_head_rows + m) * 64 +
                                (c & 3) * 16
                          : reinterpret_cast<const uint8_t*>(p.x) + (size_t)m * pitch + c * 16;
    } else {
      const int row = 8 * (g - XI) + (lane >> 3);
      src[i] = reinterpret_cast<const uint8_t*>(p.w) + (size_t)(n0 + row) * pitch + swz(row, lane & 7) * 16;
    }
  }
  const uint32_t lds0 = lds_addr_of(smem);
  auto issue_part = [&](int kt, int buf, int i0, int i1) {
#pragma unroll
    for (int i = 0; i < LPS; ++i) {
      if (i < i0 || i >= i1) continue;
      const uint32_t la = lds0 + buf * kStage + (wave + i * 4) * 1024;
      lds_dma16(src[i] + (size_t)kt * (i < XL ? x_stage : (size_t)kRowBytes), __builtin_amdgcn_readfirstlane(la));
    }
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;

#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < KT) issue_part(st, st, XL, LPS);
  wait_inputs();
  issue_epilogue_operands<BM, BN, E, LN, 4>(p, m0, n0, M, epi, wave, lane);
#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < KT) issue_part(st, st, 0, XL);

  for (int kt0 = 0; kt0 < KT; kt0 += STAGES) {
#pragma unroll
    for (int u = 0; u < STAGES; ++u) {
      const int kt = kt0 + u;
      if (kt < KT) {
        // stage 0: everything requested so far; later stages: the usual ring
        if (kt == 0)
          wait_vmcnt<0>();
        else
          wait_stage<LPS, STAGES - 2>(min(STAGES - 2, KT - 1 - kt));
        __syncthreads();  // stage kt visible to all waves; buffer of stage kt-1 is free
        const uint8_t* xs = smem + u * kStage;
        const uint8_t* ws = xs + BM * kRowBytes;
        bf16x8_t af[4][TN], bfr[4][TM];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
          for (int tn = 0; tn < TN; ++tn) {
            const int r = wn * WN + tn * 32 + l32;
            af[q][tn] = as_bf16x8(ld16(ws + r * kRowBytes + swz(r, 2 * q + half) * 16));
          }
#pragma unroll
          for (int tm = 0; tm < TM; ++tm) {
            const int r = wm * WM + tm * 32 + l32;
            bfr[q][tm] = as_bf16x8(ld16(xs + r * kRowBytes + swz(r, 2 * q + half) * 16));
          }
        }
        if (kt + STAGES - 1 < KT) issue_part(kt + STAGES - 1, (u + STAGES - 1) % STAGES, 0, LPS);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int tm = 0; tm < TM; ++tm)
#pragma unroll
            for (int tn = 0; tn < TN; ++tn)
              acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[q][tn], bfr[q][tm], acc[tm][tn], 0, 0, 0);
      }
    }
  }
  constexpr int NRB = BM * (BN * 4 + 16) <= STAGES * kStage ? 1 : 2;
  store_tile<BM, BN, bf16_t, Quant::None, E, TM, TN, NRB, 1, LN, true>(acc, smem, p, m0, n0, M, epi);
}

// LDS use of each item kind (after the block state).
constexpr int kLdsO = gemm_item_ring_bytes<64, 64, 4>() +
                      epi_layout(64, 64, true, false, true, kPipeHidden, kPipeHidden).bytes;
constexpr int kLdsU = gemm_item_ring_bytes<64, kUpCols, 3>() +
                      epi_layout(64, kUpCols, false, true, false, kPipeHidden, kPipeHidden).bytes;
constexpr int kLdsA = qkv_attention_ring_bytes<2>() + kFVecBytes + kFStatBytes;
static_assert(kLdsO <= kPItemBytes && kLdsU <= kPItemBytes && kLdsA <= kPItemBytes, "item LDS");

// ---------------------------------------------------------------------------
// Embedding item: rows r .. r+15 of this XCD, four per wave, each
// LN(word[id] + pos[s] + type[0]) stored as bf16.  The row -> (sequence,
// position) map comes from the mask (the j-th real token of its sequence), so
// masks with holes work; every load of the wave's four rows is issued at once.
// ---------------------------------------------------------------------------
__device__ __attribute__((noinline)) void embed_item(const PipeParams& p, const PipeState& S, int r_begin) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int H = p.H, nch = H / 8;
  const int Sq = p.S;
  constexpr int R = kEmbRows / 4;
  int g[R], b[R], jpos[R];
  bool live[R];
#pragma unroll
  for (int j = 0; j < R; ++j) {
    g[j] = S.row0 + r_begin + wave + 4 * j;
    live[j] = g[j] < S.row1;
    b[j] = live[j] ? seq_of_row(S, g[j]) : S.seq0;
    jpos[j] = live[j] ? g[j] - S.cu[b[j]] : 0;
  }
  // mask bytes: positions lane and lane + 64 of each row's sequence
  uint8_t mk[R][2];
#pragma unroll
  for (int j = 0; j < R; ++j)
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      const int s = lane + 64 * h2;
      mk[j][h2] = live[j] && s < Sq ? p.mask[(size_t)b[j] * Sq + s] : 0;
    }
  int pos[R];
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const uint64_t b0 = __ballot(mk[j][0] != 0), b1 = __ballot(mk[j][1] != 0);
    const int c0 = __popcll(b0);
    const uint64_t bal = jpos[j] < c0 ? b0 : b1;
    const int want = jpos[j] < c0 ? jpos[j] : jpos[j] - c0;
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    const bool hit = ((bal >> lane) & 1ull) && __popcll(bal & below) == want;
    const uint64_t hb = __ballot(hit);
    pos[j] = hb ? (__ffsll((long long)hb) - 1) + (jpos[j] < c0 ? 0 : 64) : 0;
  }
  int id[R];
#pragma unroll
  for (int j = 0; j < R; ++j) id[j] = live[j] ? min(max(p.ids[(size_t)b[j] * Sq + pos[j]], 0), p.vocab - 1) : 0;
  const int ch = min(lane, nch - 1);
  uint4 rw[R], rp[R];
  const uint4 rt = *reinterpret_cast<const uint4*>(p.type + ch * 8);
#pragma unroll
  for (int j = 0; j < R; ++j) {
    rw[j] = *reinterpret_cast<const uint4*>(p.word + (size_t)id[j] * H + ch * 8);
    rp[j] = *reinterpret_cast<const uint4*>(p.pos + (size_t)pos[j] * H + ch * 8);
  }
  float gm[8], bt[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    gm[e] = p.emb_g[ch * 8 + e];
    bt[e] = p.emb_b[ch * 8 + e];
  }
  const float t8[8] = {__uint_as_float(rt.x << 16), __uint_as_float(rt.x & 0xffff0000u),
                       __uint_as_float(rt.y << 16), __uint_as_float(rt.y & 0xffff0000u),
                       __uint_as_float(rt.z << 16), __uint_as_float(rt.z & 0xffff0000u),
                       __uint_as_float(rt.w << 16), __uint_as_float(rt.w & 0xffff0000u)};
#pragma unroll
  for (int j = 0; j < R; ++j) {
    if (!live[j]) continue;  // wave-uniform
    const uint32_t a[4] = {rw[j].x, rw[j].y, rw[j].z, rw[j].w}, c[4] = {rp[j].x, rp[j].y, rp[j].z, rp[j].w};
    float v[8], sum = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(a[i] << 16) + __uint_as_float(c[i] << 16) + t8[2 * i];
      v[2 * i + 1] = __uint_as_float(a[i] & 0xffff0000u) + __uint_as_float(c[i] & 0xffff0000u) + t8[2 * i + 1];
    }
    const bool in = lane < nch;
#pragma unroll
    for (int e = 0; e < 8; ++e) sum += in ? v[e] : 0.0f;
    const float mean = wave_sum(sum) / (float)H;
    float sq = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) sq += in ? (v[e] - mean) * (v[e] - mean) : 0.0f;
    const float rstd = 1.0f / sqrtf(wave_sum(sq) / (float)H + p.eps);
    if (in) {
      float o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (v[e] - mean) * rstd * gm[e] + bt[e];
      *reinterpret_cast<uint4*>(p.X + (size_t)g[j] * H + lane * 8) =
          make_uint4(pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]), pack_bf16x2(o[4], o[5]),
                     pack_bf16x2(o[6], o[7]));
    }
  }
}

// ---------------------------------------------------------------------------
// Pooling item: sequence b's rows are the last layer's LN2 inputs with their
// partial statistics; average (x - mean) * rstd over the rows, apply gamma and
// beta, then divide by max(||.||_2, 1e-12).  A sequence without tokens gives
// the zero vector.  Wave w takes rows w, w + 4, ...; kPoolBatch rows are in
// flight per wave; lanes 0..15 each merge one row's statistics.
// ---------------------------------------------------------------------------
__device__ __attribute__((noinline)) void pool_item(const PipeParams& p, const PipeState& S, int b, uint8_t* lds) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int H = p.H, nch = H / 8, np = H >> 6;
  const int r0 = uni(S.cu[b]), L = uni(S.cu[b + 1]) - r0;
  float* part = reinterpret_cast<float*>(lds);  // [4][H]
  float* red = part + 4 * H;                    // [4]
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
  const int ch = min(lane, nch - 1);
  for (int rb = wave; rb < L; rb += 4 * kPoolBatch) {
    uint4 raw[kPoolBatch];
#pragma unroll
    for (int k = 0; k < kPoolBatch; ++k) {
      const int r = min(rb + 4 * k, L - 1);  // rows past the end: loaded, not added
      raw[k] = *reinterpret_cast<const uint4*>(p.X + (size_t)(r0 + r) * H + ch * 8);
    }
    // lane k < kPoolBatch: statistics of row rb + 4k
    float2 st = make_float2(0.0f, 1.0f);
    if (lane < kPoolBatch) st = row_ln_stats(p.S2 + (size_t)(r0 + min(rb + 4 * lane, L - 1)) * np, np, p.eps);
#pragma unroll
    for (int k = 0; k < kPoolBatch; ++k) {
      const float mean = __shfl(st.x, k, 64), rstd = __shfl(st.y, k, 64);
      if (rb + 4 * k < L) {
        const uint32_t w[4] = {raw[k].x, raw[k].y, raw[k].z, raw[k].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[2 * i] += (__uint_as_float(w[i] << 16) - mean) * rstd;
          acc[2 * i + 1] += (__uint_as_float(w[i] & 0xffff0000u) - mean) * rstd;
        }
      }
    }
  }
  if (lane < nch)
#pragma unroll
    for (int e = 0; e < 8; ++e) part[wave * H + lane * 8 + e] = acc[e];
  __syncthreads();
  const float inv_l = 1.0f / fmaxf((float)L, 1e-9f);
  float val[2] = {0.0f, 0.0f}, ss = 0.0f;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int c = tid + 256 * k;
    if (c < H && L > 0) {
      const float m = (part[c] + part[H + c] + part[2 * H + c] + part[3 * H + c]) * inv_l;
      val[k] = fmaf(p.last_g[c], m, p.last_b[c]);
      ss += val[k] * val[k];
    }
  }
  ss = wave_sum(ss);
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  const float inv = 1.0f / fmaxf(sqrtf(red[0] + red[1] + red[2] + red[3]), 1e-12f);
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int c = tid + 256 * k;
    if (c < H) p.out[(size_t)b * H + c] = val[k] * inv;
  }
}

// The layer items, each its own function (its own register allocation): the
// kernel's register budget is the largest of them, not their union.
__device__ __attribute__((noinline)) void attention_item(const PipeParams& p, int l, int row0, int len, int h,
                                                         uint8_t* ilds, DepWait dw) {
  l = uni(l);
  const PipeLayer& W = uni_ptr(p.layers)[l];
  FusedAttnParams fa{};
  fa.x = p.X; fa.wqkv = W.wqkv; fa.bqkv = W.bqkv; fa.fold_u = W.uq;
  fa.x_stats = l > 0 ? p.S2 : nullptr; fa.ln_eps = p.eps;
  fa.out = p.CTX; fa.out_rows = uni(p.ctx_rows); fa.H = uni(p.H); fa.heads = uni(p.heads); fa.scale = p.scale;
  uint8_t* vec = ilds + qkv_attention_ring_bytes<2>();
  qkv_attention_block<2>(fa, uni(row0), uni(len), uni(h), ilds, reinterpret_cast<float*>(vec),
                         reinterpret_cast<float2*>(vec + kFVecBytes), dw);
}

__device__ __forceinline__ GemmParams item_params(const PipeParams& p, int row_end) {
  GemmParams g{};
  g.M = row_end;
  g.dtype = DType::BF16;
  g.quant = Quant::None;
  g.ln_eps = p.eps;
  return g;
}

// output projection + bias + residual, and LN1's statistics of its output
__device__ __attribute__((noinline)) void out_proj_item(const PipeParams& p, int l, int row_end, int m0, int n0,
                                                        uint8_t* ilds, DepWait dw) {
  l = uni(l);
  const PipeLayer& W = uni_ptr(p.layers)[l];
  GemmParams g = item_params(p, uni(row_end));
  g.x = p.CTX; g.x_head_rows = p.ctx_rows; g.w = W.wo; g.bias = W.bo;
  g.residual = p.X; g.y = p.A; g.y_stats = p.S1; g.N = p.H; g.K = p.H; g.epi = Epi::BiasResidual;
  if (l == 0) {
    gemm_item<64, 64, 4, Epi::BiasResidual, kLnOut>(g, ilds, m0, n0, dw);
  } else {  // the residual is the previous layer's LN2 input
    g.res_stats = p.S2; g.res_gamma = W.res_g; g.res_beta = W.res_b;
    gemm_item<64, 64, 4, Epi::BiasResidual, kLnRes | kLnOut>(g, ilds, m0, n0, dw);
  }
}

// FFN-up on LN1 (folded into W1) + bias + erf-GELU
__device__ __attribute__((noinline)) void ffn_up_item(const PipeParams& p, int l, int row_end, int m0, int n0,
                                                      uint8_t* ilds, DepWait dw) {
  l = uni(l);
  const PipeLayer& W = uni_ptr(p.layers)[l];
  GemmParams g = item_params(p, uni(row_end));
  g.x = p.A; g.x_stats = p.S1; g.fold_u = W.u1; g.w = W.w1; g.bias = W.v1;
  g.y = p.G; g.N = p.F; g.K = p.H; g.epi = Epi::BiasGelu;
  gemm_item<64, kUpCols, 3, Epi::BiasGelu, kLnX>(g, ilds, m0, n0, dw);
}

// FFN-down + bias + LN1(residual), and LN2's statistics of its output
__device__ __attribute__((noinline)) void ffn_down_item(const PipeParams& p, int l, int row_end, int m0, int n0,
                                                        uint8_t* ilds, DepWait dw) {
  l = uni(l);
  const PipeLayer& W = uni_ptr(p.layers)[l];
  GemmParams g = item_params(p, uni(row_end));
  g.x = p.G; g.w = W.w2; g.bias = W.b2;
  g.residual = p.A; g.res_stats = p.S1; g.res_gamma = W.ln1_g; g.res_beta = W.ln1_b;
  g.y = p.X; g.y_stats = p.S2; g.N = p.H; g.K = p.F; g.epi = Epi::BiasResidual;
  gemm_item<64, 64, 4, Epi::BiasResidual, kLnRes | kLnOut>(g, ilds, m0, n0, dw);
}

__global__ __launch_bounds__(kPThreads, 2) void encoder_pipe_kernel(PipeParams params) {
  // The item functions read the parameters where the launch put them (the
  // kernel-argument segment, `params` is the only argument): a reference to
  // the by-value argument would make the compiler copy it to scratch memory.
  const PipeParams& p = *(const PipeParams*)__builtin_amdgcn_kernarg_segment_ptr();
  (void)params;
  extern __shared__ __attribute__((aligned(1024))) uint8_t plds[];
  PipeState& S = *reinterpret_cast<PipeState*>(plds);
  uint8_t* ilds = plds + kPStateBytes;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int xcd = xcc_id();
  int* sy = p.sync + (size_t)xcd * kPipeSyncStride;

  // 1. Token counts of every sequence, then their prefix: the compact row
  //    offsets.  Rows that are whole 16-byte chunks are counted a chunk per
  //    thread, others a row per wave (a ballot per 64 positions).
  const int B = p.B, Sq = p.S;
  for (int b = tid; b <= B; b += kPThreads) S.cu[b] = 0;
  __syncthreads();
  if (Sq % 16 != 0 || (reinterpret_cast<uintptr_t>(p.mask) & 15) != 0) {
    for (int b = wave; b < B; b += kPThreads / 64) {
      const bool v0 = lane < Sq && p.mask[(size_t)b * Sq + lane] != 0;
      const bool v1 = lane + 64 < Sq && p.mask[(size_t)b * Sq + lane + 64] != 0;
      const int n = __popcll(__ballot(v0)) + __popcll(__ballot(v1));
      if (lane == 0) S.cu[b] = n;
    }
  } else {
    const int chunks = B * Sq / 16;
    for (int c = tid; c < chunks; c += kPThreads) {
      const uint4 u = *reinterpret_cast<const uint4*>(p.mask + (size_t)c * 16);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
      int n = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        uint32_t t = w[k] | (w[k] >> 4);
        t |= t >> 2;
        t |= t >> 1;
        n += __popc(t & 0x01010101u);
      }
      if (n) atomicAdd(&S.cu[c * 16 / Sq], n);
    }
  }
  __syncthreads();
  if (wave == 0) {
    int carry = 0;
    for (int c0 = 0; c0 < B; c0 += 64) {
      const int v = c0 + lane < B ? S.cu[c0 + lane] : 0;
      int incl = v;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int n = __shfl_up(incl, o, 64);
        if (lane >= o) incl += n;
      }
      if (c0 + lane < B) S.cu[c0 + lane] = carry + incl - v;
      carry += __shfl(incl, 63, 64);
    }
    if (lane == 0) S.cu[B] = carry;
  }
  __syncthreads();
  // 2. This XCD's run of sequences: the boundaries are the sequence starts
  //    nearest to x * T / 8.
  const int H = p.H, F = p.F, L = p.L, heads = p.heads;
  const int ctO = H / 64, ctU = F / kUpCols, ctD = H / 64;
  if (tid == 0) {
    const int T = S.cu[B];
    // boundary x: the first b with cu[b] >= x T / 8, or the one before it when
    // that start is nearer -- non-decreasing in x, so the runs never overlap
    auto cut = [&](int x) {
      if (x <= 0) return 0;
      if (x >= 8) return B;
      const int target = (int)(((long long)x * T + 4) / 8);
      int lo = 0, hi = B;  // lower bound of target in cu[0..B]
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (S.cu[mid] < target) lo = mid + 1;
        else hi = mid;
      }
      return (lo > 0 && target - S.cu[lo - 1] < S.cu[lo] - target) ? lo - 1 : lo;
    };
    const int s0 = cut(xcd), s1 = max(cut(xcd + 1), s0);
    S.seq0 = s0;
    S.seq1 = s1;
    S.row0 = S.cu[s0];
    S.row1 = S.cu[s1];
    const int nrows = S.row1 - S.row0;
    S.nrt = (nrows + kRowTile - 1) / kRowTile;
    const int nseq = s1 - s0;
    S.total = (nrows + kEmbRows - 1) / kEmbRows + L * (nseq * heads + S.nrt * (ctO + ctU + ctD)) + nseq;
  }
  __syncthreads();
  const int seq0 = uni(S.seq0), seq1 = uni(S.seq1), row0 = uni(S.row0), row1 = uni(S.row1);
  const int total = uni(S.total);
  const int nseq = seq1 - seq0, nrt = uni(S.nrt), nrows = row1 - row0;
  const int nE = (nrows + kEmbRows - 1) / kEmbRows;
  const int nA = nseq * heads, nO = nrt * ctO, nU = nrt * ctU, nD = nrt * ctD;
  const int per_layer = nA + nO + nU + nD;

  // sequences -> row tiles (XCD-relative) and back
  auto rt_range_of_seq = [&](int b, int& lo, int& hi) {
    lo = uni((S.cu[b] - row0) / kRowTile);
    hi = uni((S.cu[b + 1] - 1 - row0) / kRowTile);
  };

  // 3. Items.  Each iteration has exactly one single-lane region, between two
  //    barriers: thread 0 counts the item just finished (its stores are
  //    complete: every wave drained its memory counters before the first
  //    barrier) and takes the next one.  Keeping the two atomics in one region
  //    with a barrier on either side stops the compiler from merging them
  //    across the loop's back edge into a loop that lane 0 and the other lanes
  //    leave at different times -- which would run a barrier a different
  //    number of times in wave 0 than in the other waves.
  int done_idx = -1;  // completion counter of the previous item
  for (;;) {
    __syncthreads();
    if (tid == 0) {
      if (done_idx >= 0) __hip_atomic_fetch_add(sy + done_idx, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      S.item = atomicAdd(sy + kQueue, 1);
    }
    __syncthreads();
    const int it = uni(S.item);
    if (it >= total) break;
    if (it < nE) {
      finish_wait();  // (no inputs: keeps the barrier count uniform)
      embed_item(p, S, it * kEmbRows);
      done_idx = kCntE;
    } else if (it - nE >= L * per_layer) {  // pooling of one sequence, after its row tiles' last FFN-down
      const int b = seq0 + (it - nE - L * per_layer);
      DepWait dw{sy, 0, -1, 0};
      if (uni(S.cu[b + 1]) > uni(S.cu[b])) {
        int lo, hi;
        rt_range_of_seq(b, lo, hi);
        dw = DepWait{sy, cnt_tile(2, L, L - 1, lo), cnt_tile(2, L, L - 1, hi), ctD};
      }
      dw();
      pool_item(p, S, b, ilds);
      done_idx = kCntP;  // (counted, not waited on)
    } else {
      int k = it - nE;
      const int l = k / per_layer;
      k -= l * per_layer;
      if (k < nA) {  // QKV projection + attention of (sequence, head)
        const int b = seq0 + k / heads, h = k % heads;
        const int r0 = uni(S.cu[b]), len = uni(S.cu[b + 1]) - r0;
        if (len > 0) {
          DepWait dw{sy, kCntE, kCntE, nE};  // layer 0: the embedding
          if (l > 0) {
            int lo, hi;
            rt_range_of_seq(b, lo, hi);
            dw = DepWait{sy, cnt_tile(2, L, l - 1, lo), cnt_tile(2, L, l - 1, hi), ctD};
          }
          attention_item(p, l, r0, len, h, ilds, dw);
        }
        done_idx = cnt_a(l, b - seq0);
      } else if (k < nA + nO) {  // after every head of every sequence in the row tile
        const int rt = (k - nA) / ctO, ct = (k - nA) % ctO;
        const int m0 = row0 + rt * kRowTile;
        const int s_lo = uni(seq_of_row(S, m0)), s_hi = uni(seq_of_row(S, min(m0 + kRowTile, row1) - 1));
        out_proj_item(p, l, row1, m0, ct * 64, ilds, DepWait{sy, cnt_a(l, s_lo - seq0), cnt_a(l, s_hi - seq0), heads});
        done_idx = cnt_tile(0, L, l, rt);
      } else if (k < nA + nO + nU) {  // after the row tile's output projection
        const int rt = (k - nA - nO) / ctU, ct = (k - nA - nO) % ctU;
        ffn_up_item(p, l, row1, row0 + rt * kRowTile, ct * kUpCols, ilds,
                    DepWait{sy, cnt_tile(0, L, l, rt), cnt_tile(0, L, l, rt), ctO});
        done_idx = cnt_tile(1, L, l, rt);
      } else {  // after the row tile's FFN-up
        const int rt = (k - nA - nO - nU) / ctD, ct = (k - nA - nO - nU) % ctD;
        ffn_down_item(p, l, row1, row0 + rt * kRowTile, ct * 64, ilds,
                      DepWait{sy, cnt_tile(1, L, l, rt), cnt_tile(1, L, l, rt), ctU});
        done_idx = cnt_tile(2, L, l, rt);
      }
    }
    done_idx = uni(done_idx);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's stores of the item are complete in L2
  }

}

// Zeroes the sync words a launch of B sequences of S tokens and L layers can
// use: block x clears XCD x's queue and abort words, its E / P counters, the
// head counters of B sequences and the tile counters of ceil(B S / 64) row
// tiles per layer.  (The sticky error word is left for rlx_encoder_check.)
__global__ __launch_bounds__(256) void pipe_clear_kernel(int* sync, int L, int B, int rts) {
  int* sy = sync + (size_t)blockIdx.x * kPipeSyncStride;
  const int t = threadIdx.x;
  if (t < kCntBase && t != kErr) sy[t] = 0;
  for (int i = t; i < L * B; i += 256) sy[cnt_a(i / B, i % B)] = 0;
  for (int i = t; i < 3 * L * rts; i += 256) {
    const int which = i / (L * rts), rem = i % (L * rts);
    sy[cnt_tile(which, L, rem / rts, rem % rts)] = 0;
  }
}

}  // namespace

bool pipe_supported(const PipeShape& s) {
  return s.H == kPipeHidden && s.heads * 32 == s.H && s.F % kUpCols == 0 && s.B >= 1 && s.B <= kPipeMaxBatch &&
         s.S >= 1 && s.S <= 128 && (long long)s.B * s.S <= kPipeMaxTokens && s.L >= 1;
}

size_t pipe_sync_bytes() { return (size_t)8 * kPipeSyncStride * sizeof(int); }

hipError_t init_pipe_attributes() {
  static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(encoder_pipe_kernel),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, kPipeLdsBytes);
  return attr;
}

hipError_t launch_encoder_pipe(const PipeParams& p, int grid, hipStream_t s) {
  const hipError_t attr = init_pipe_attributes();
  if (attr != hipSuccess) return attr;
  if (grid <= 0 || p.L > kPipeMaxLayers || !pipe_supported(PipeShape{p.B, p.S, p.H, p.F, p.heads, p.L}))
    return hipErrorInvalidValue;
  const int rts = (p.B * p.S + 63) / 64;
  hipLaunchKernelGGL(pipe_clear_kernel, dim3(8), dim3(256), 0, s, p.sync, p.L, p.B, rts);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  RLX_LOG_LAUNCH("encoder_pipe_kernel", dim3(grid), dim3(kPThreads), kPipeLdsBytes, "persistent B=%d S=%d layers=%d",
                 p.B, p.S, p.L);
  hipLaunchKernelGGL(encoder_pipe_kernel, dim3(grid), dim3(kPThreads), kPipeLdsBytes, s, p);
  return hipGetLastError();
}

}  // namespace rlx
