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

// The mask scan keeps kScanLoads mask loads per lane in flight: a wave takes
// kScanLoads / NCH sequences at a time, NCH 64-position loads each (NCH the
// row length in 64s rounded up to a power of two, S <= 64 * kScanMaxChunks).
constexpr int kScanLoads = 32;
constexpr int kScanMaxChunks = 8;

// Mask bytes of sequences b0 .. b0 + SEQS - 1 at positions 64 c + lane, 0
// past the batch or the row.  Every load is issued unconditionally at an
// in-bounds (clamped) address and selected afterwards: a load under a
// per-lane condition gets its own wait for the data, which serialises them.
// Needs B >= 1 and 1 <= S <= 64 * NCH.
template <int SEQS, int NCH>
__device__ __forceinline__ void load_mask_group(const uint8_t* mask, int B, int S, int b0, int lane,
                                                uint8_t (&mb)[SEQS][NCH]) {
  uint8_t raw[SEQS][NCH];
#pragma unroll
  for (int g = 0; g < SEQS; ++g)
#pragma unroll
    for (int c = 0; c < NCH; ++c) raw[g][c] = mask[(size_t)min(b0 + g, B - 1) * S + min(64 * c + lane, S - 1)];
#pragma unroll
  for (int g = 0; g < SEQS; ++g)
#pragma unroll
    for (int c = 0; c < NCH; ++c) mb[g][c] = (b0 + g < B && 64 * c + lane < S) ? raw[g][c] : 0;
}

template <int NCH>
__global__ __launch_bounds__(1024) void mask_scan_kernel(const uint8_t* mask, int B, int S, int* cu, int* tok_src,
                                                         int* tok_dst, int* order, int2* rank_rows) {
  constexpr int SEQS = kScanLoads / NCH;
  extern __shared__ int offs[];  // [B+1]: token counts, then their exclusive prefix; then [B] ranks (with order)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const uint64_t below = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
  // Each wave takes SEQS sequences at a time and requests all their mask
  // bytes before the first ballot: one memory round trip per group.  The
  // wave's first group stays in registers for the second pass (the only
  // group when B <= 16 * SEQS, e.g. 256 sequences of <= 128 positions).
  const int first = wave * SEQS, stride = nw * SEQS;
  uint8_t mb0[SEQS][NCH];
  auto count = [&](int b0, const uint8_t (&mb)[SEQS][NCH]) {
#pragma unroll
    for (int g = 0; g < SEQS; ++g) {
      int cnt = 0;
#pragma unroll
      for (int c = 0; c < NCH; ++c) cnt += __popcll(__ballot(mb[g][c] != 0));
      if (lane == 0 && b0 + g < B) offs[b0 + g] = cnt;
    }
  };
  if (first < B) {
    load_mask_group<SEQS, NCH>(mask, B, S, first, lane, mb0);
    count(first, mb0);
  }
  for (int b0 = first + stride; b0 < B; b0 += stride) {
    uint8_t mb[SEQS][NCH];
    load_mask_group<SEQS, NCH>(mask, B, S, b0, lane, mb);
    count(b0, mb);
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
  if (order && rank_rows) {  // the ranks are still in LDS after the prefix
    const int* rank = offs + B + 1;
    for (int i = threadIdx.x; i < B; i += blockDim.x) rank_rows[rank[i]] = make_int2(offs[i], offs[i + 1] - offs[i]);
  }
  auto emit = [&](int b0, const uint8_t (&mb)[SEQS][NCH]) {
#pragma unroll
    for (int g = 0; g < SEQS; ++g) {
      const int b = b0 + g;
      if (b >= B) break;  // wave-uniform
      int base = offs[b];
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const int s = 64 * c + lane;
        const bool v = mb[g][c] != 0;
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
  };
  if (first < B) emit(first, mb0);
  for (int b0 = first + stride; b0 < B; b0 += stride) {
    uint8_t mb[SEQS][NCH];
    load_mask_group<SEQS, NCH>(mask, B, S, b0, lane, mb);
    emit(b0, mb);
  }
}

// Row held by one wave as 16-byte chunks: lane owns chunks lane, lane+64, ...
// (EPC elements each), so every wave-wide load or store is one contiguous run.
template <typename T> struct Chunk;
template <> struct Chunk<bf16_t> {
  static constexpr int EPC = 8;
  static __device__ __forceinline__ void load(const bf16_t* p, float v[8]) {
    from_raw(*reinterpret_cast<const uint4*>(p), v);
  }
  static __device__ __forceinline__ void from_raw(uint4 u, float v[8]) {
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
    from_raw(*reinterpret_cast<const uint4*>(p), v);
  }
  static __device__ __forceinline__ void from_raw(uint4 u, float v[4]) {
    v[0] = __uint_as_float(u.x); v[1] = __uint_as_float(u.y); v[2] = __uint_as_float(u.z); v[3] = __uint_as_float(u.w);
  }
  static __device__ __forceinline__ void store(float* p, const float v[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
};

// Chunks per lane: H <= 1024 gives at most 2 (bf16) or 4 (f32).
template <typename T> constexpr int kMaxCpl = 8 / Chunk<T>::EPC * 2;

// gamma and beta of the columns a lane's chunks hold (chunk lane + 64 i),
// loaded with the row they scale instead of after its reductions: one
// memory round trip less per row.  Every lane loads NC chunks, clamped to
// the last one (lanes past the row's end load a copy they never use), so the
// loads cannot be sunk into the branches that use them.
template <typename T, int NC = kMaxCpl<T>>
struct LnAffine {
  float g[NC][Chunk<T>::EPC], b[NC][Chunk<T>::EPC];
  __device__ __forceinline__ void load(const float* gamma, const float* beta, int H) {
    constexpr int EPC = Chunk<T>::EPC;
    const int lane = threadIdx.x & 63;
    const int nch = H / EPC;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int ch = min(lane + 64 * i, nch - 1);
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        g[i][e] = gamma[ch * EPC + e];
        b[i][e] = beta[ch * EPC + e];
      }
    }
  }
};

// LayerNorm of the wave's row held in v (fp32), written as T when `keep`,
// with the lane's gamma and beta already in registers.  The norm is computed
// either way, so that a caller's loads of the row are never sunk into the
// branch of the store (the reductions are cross-lane and stay outside it).
template <typename T, int NC = kMaxCpl<T>>
__device__ __forceinline__ void ln_row_store(float (&v)[NC][Chunk<T>::EPC], int H, const LnAffine<T, NC>& aff,
                                             float eps, T* out, bool keep = true) {
  constexpr int EPC = Chunk<T>::EPC, CPL = NC;
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
      for (int e = 0; e < EPC; ++e) o[e] = (v[i][e] - mean) * rstd * aff.g[i][e] + aff.b[i][e];
      if (keep) Chunk<T>::store(out + ch * EPC, o);
    }
  }
}

template <typename T, int NC>
__global__ __launch_bounds__(256) void embed_ln_kernel(const int* ids, const T* word, const T* pos, const T* type,
                                                       const float* gamma, const float* beta, float eps, int vocab,
                                                       int S, int H, const int* tok_src, const int* n_dev, int n_max,
                                                       T* x) {
  constexpr int EPC = Chunk<T>::EPC;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_max) return;
  // the token count, the token's source and the LayerNorm affine in one
  // round trip (tok_src holds n_max entries; past the count it is unused)
  LnAffine<T, NC> aff;
  aff.load(gamma, beta, H);
  const int src = tok_src[t];
  const int n = min(n_max, *n_dev);
  if (t >= n) return;
  const int lane = threadIdx.x & 63;
  const int s = src % S;
  const int id = min(max(ids[src], 0), vocab - 1);
  const int nch = H / EPC;
  float v[NC][EPC];
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int ch = min(lane + 64 * i, nch - 1);
    float a[EPC], b[EPC], c[EPC];
    Chunk<T>::load(word + (size_t)id * H + ch * EPC, a);
    Chunk<T>::load(pos + (size_t)s * H + ch * EPC, b);
    Chunk<T>::load(type + ch * EPC, c);
#pragma unroll
    for (int e = 0; e < EPC; ++e) v[i][e] = a[e] + b[e] + c[e];
  }
  ln_row_store<T, NC>(v, H, aff, eps, x + (size_t)t * H);
}

// Mask scan fused with the embedding gather + LayerNorm, for small masks
// (B*S <= kEmbedScanMaxMask, B <= kMaxOrderedBatch).  Block (b, p) embeds the
// real tokens p*16 .. p*16+15 of sequence b, four per wave.  Every block
// first counts the real tokens of all sequences itself (the whole mask is at
// most 16 KB), so it knows its sequence's offset without waiting on another
// block; block (b, 0) also writes the scan's outputs for sequence b: cu[b]
// (and cu[B] for the last sequence), the token maps of row b and the
// sequence's place in the longest-first order.  One launch and one memory
// round trip less than the mask scan followed by the embedding kernel.
constexpr int kEmbedScanTokens = 16;  // real tokens per block
template <typename T, int NC>
__global__ __launch_bounds__(256) void embed_scan_kernel(const uint8_t* mask, const int* ids, int B, int S,
                                                         const T* word, const T* pos, const T* type,
                                                         const float* gamma, const float* beta, float eps, int vocab,
                                                         int H, int* cu, int* tok_src, int* tok_dst, int* order,
                                                         T* x, int2* rank_rows) {
  constexpr int EPC = Chunk<T>::EPC, CPL = NC;  // chunks per lane: NC * 64 * EPC >= H
  __shared__ __attribute__((aligned(16))) uint8_t mlds[kEmbedScanMaxMask];  // the whole mask
  __shared__ int cnt[kMaxOrderedBatch];
  __shared__ int posl[kEmbedScanMaxSeq];  // positions of sequence b's real tokens
  __shared__ int idl[kEmbedScanMaxSeq];   // token ids of sequence b
  const int b = blockIdx.x, p = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t below = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
  // One round trip for the mask (16-byte loads when it allows them), sequence
  // b's ids (the rows' gather needs them only after the scan has placed the
  // tokens) and the LayerNorm affine: every load issued before any is
  // waited for, then the mask and ids go to LDS.  Loads and LDS stores are
  // unconditional, at indexes clamped into the arrays (lanes past the end
  // copy the last element again, to the same place): a load used only under
  // a condition is sunk into that branch and waited for there, one at a time.
  const int nm = B * S;
  constexpr int MJ = kEmbedScanMaxMask / (16 * 256), IJ = kEmbedScanMaxSeq / 256;
  int ir[IJ];
  LnAffine<T, NC> aff;
  auto load_ids_affine = [&] {
#pragma unroll
    for (int j = 0; j < IJ; ++j) ir[j] = ids[(size_t)b * S + min((int)threadIdx.x + 256 * j, S - 1)];
    aff.load(gamma, beta, H);
  };
  if ((reinterpret_cast<uintptr_t>(mask) & 15) == 0 && (nm & 15) == 0) {
    uint4 mr[MJ];
#pragma unroll
    for (int j = 0; j < MJ; ++j)
      mr[j] = *reinterpret_cast<const uint4*>(mask + min((int)(threadIdx.x + 256 * j) * 16, nm - 16));
    load_ids_affine();
#pragma unroll
    for (int j = 0; j < MJ; ++j)
      *reinterpret_cast<uint4*>(mlds + min((int)(threadIdx.x + 256 * j) * 16, nm - 16)) = mr[j];
  } else {
    load_ids_affine();
#pragma unroll 16
    for (int j = 0; j < kEmbedScanMaxMask / 256; ++j) {
      const int i = threadIdx.x + 256 * j;
      if (i < nm) mlds[i] = mask[i];
    }
  }
#pragma unroll
  for (int j = 0; j < IJ; ++j) idl[min((int)threadIdx.x + 256 * j, S - 1)] = ir[j];
  __syncthreads();
  // real tokens of every sequence
  if ((S & 15) == 0) {
    // one thread per sequence, 16 bytes at a time (rows start 16-byte aligned
    // in LDS): the non-zero bytes of a word are counted by folding each byte's
    // bits into its lowest bit
    for (int q = threadIdx.x; q < B; q += 256) {
      int c = 0;
      for (int i = 0; i < S; i += 16) {
        const uint4 u = *reinterpret_cast<const uint4*>(mlds + q * S + i);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          uint32_t t = w[k] | (w[k] >> 4);
          t |= t >> 2;
          t |= t >> 1;
          c += __popc(t & 0x01010101u);
        }
      }
      cnt[q] = c;
    }
  } else {
    // one wave per sequence, a ballot per 64 positions
    for (int q = wave; q < B; q += 4) {
      int c = 0;
      for (int s0 = 0; s0 < S; s0 += 64) c += __popcll(__ballot(s0 + lane < S && mlds[q * S + s0 + lane] != 0));
      if (lane == 0) cnt[q] = c;
    }
  }
  // positions of this sequence's real tokens (wave 0), and its token maps (block p = 0)
  if (wave == 0) {
    int base = 0;
    for (int s0 = 0; s0 < S; s0 += 64) {
      const int s = s0 + lane;
      const bool v = s < S && mlds[b * S + s] != 0;
      const uint64_t bal = __ballot(v);
      if (v) posl[base + __popcll(bal & below)] = s;
      base += __popcll(bal);
    }
  }
  __syncthreads();
  const int L = cnt[b];
  int off = 0, ahead = 0;  // real tokens before sequence b; sequences placed before b in the order
  for (int q = lane; q < B; q += 64) {
    off += q < b ? cnt[q] : 0;
    ahead += (cnt[q] > L || (cnt[q] == L && q < b)) ? 1 : 0;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    off += __shfl_xor(off, o, 64);
    ahead += __shfl_xor(ahead, o, 64);
  }
  if (p == 0) {
    if (threadIdx.x == 0) {
      cu[b] = off;
      if (b == B - 1) cu[B] = off + L;
      if (order) order[ahead] = b;
      if (rank_rows) rank_rows[ahead] = make_int2(off, L);
    }
    for (int i = threadIdx.x; i < L; i += 256) tok_src[off + i] = b * S + posl[i];
    for (int s = threadIdx.x; s < S; s += 256) tok_dst[(size_t)b * S + s] = -1;
    __syncthreads();  // the real positions overwrite the -1s after them
    for (int i = threadIdx.x; i < L; i += 256) tok_dst[(size_t)b * S + posl[i]] = off + i;
  }
  // embedding rows of this block's tokens: every row of the wave's tokens
  // requested before any is used (tokens past the sequence end read row 0
  // and are not stored)
  const int nch = H / EPC;
  constexpr int TPW = kEmbedScanTokens / 4;  // tokens per wave
  int sp[TPW], id[TPW];
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    const int i = p * kEmbedScanTokens + wave + 4 * j;
    sp[j] = i < L ? posl[i] : -1;
    id[j] = sp[j] >= 0 ? min(max(idl[sp[j]], 0), vocab - 1) : 0;
  }
  uint4 rw[TPW][CPL], rp[TPW][CPL], rt[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int ch = min(lane + 64 * c, nch - 1);
    rt[c] = *reinterpret_cast<const uint4*>(type + ch * EPC);
#pragma unroll
    for (int j = 0; j < TPW; ++j) {
      rw[j][c] = *reinterpret_cast<const uint4*>(word + (size_t)id[j] * H + ch * EPC);
      rp[j][c] = *reinterpret_cast<const uint4*>(pos + (size_t)max(sp[j], 0) * H + ch * EPC);
    }
  }
  float v[TPW][CPL][EPC];
#pragma unroll
  for (int j = 0; j < TPW; ++j)
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      float a[EPC], bb[EPC], t[EPC];
      Chunk<T>::from_raw(rw[j][c], a);
      Chunk<T>::from_raw(rp[j][c], bb);
      Chunk<T>::from_raw(rt[c], t);
#pragma unroll
      for (int e = 0; e < EPC; ++e) v[j][c][e] = a[e] + bb[e] + t[e];
    }
#pragma unroll
  for (int j = 0; j < TPW; ++j)
    ln_row_store<T, NC>(v[j], H, aff, eps, x + (size_t)(off + p * kEmbedScanTokens + wave + 4 * j) * H, sp[j] >= 0);
}

template <typename T, int NC>
__global__ __launch_bounds__(256) void layer_norm_kernel(const T* a, const float* gamma, const float* beta, float eps,
                                                         int H, const int* n_dev, int n_max, T* y) {
  constexpr int EPC = Chunk<T>::EPC;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_max) return;
  // the affine in the round trip of the row count, then the row
  const int lane = threadIdx.x & 63;
  const int nch = H / EPC;
  LnAffine<T, NC> aff;
  aff.load(gamma, beta, H);
  const int n = n_dev ? min(n_max, *n_dev) : n_max;
  if (t >= n) return;
  float v[NC][EPC];
#pragma unroll
  for (int i = 0; i < NC; ++i) Chunk<T>::load(a + (size_t)t * H + min(lane + 64 * i, nch - 1) * EPC, v[i]);
  ln_row_store<T, NC>(v, H, aff, eps, y + (size_t)t * H);
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
// norm.  Each wave requests its first kPoolBatch rows before anything else,
// so their loads are in flight while the rows' LayerNorm statistics (deferred
// input) are merged, one thread per row: the two round trips overlap.  A batch
// is 16 chunks per lane (8 rows of bf16: a 128-token sequence at once).
constexpr int kMaxPoolRows = 512;    // the longest sequence
constexpr int kPoolSplitRows = 64;   // rows per block when sequences are split
constexpr int kPoolSplitAbove = 128;  // split when sequences may be longer than this
// With x_stats the rows are pre-LayerNorm values with their partial
// statistics (deferred LayerNorm): the block averages (x - mean) * rstd and
// applies gamma and beta to the average.
// Finishes a pooled row: thread c < H holds column c's sum over the
// sequence's L rows (normalised rows when deferred); the mean, the LayerNorm's
// gamma and beta of a deferred input, then the L2 normalisation over the
// block (16 waves).
// g and bt are column c's gamma and beta (used when deferred), loaded by the
// caller when its block starts so that they are not a round trip of their own.
__device__ __forceinline__ void pool_finish(float sum, int L, int H, bool deferred, bool gamma_scaled, float g,
                                            float bt, float* out_row, float* red) {
  const int c = threadIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float mean = 0.0f;
  if (c < H) {
    mean = sum / fmaxf((float)L, 1e-9f);
    if (deferred) mean = L > 0 ? (gamma_scaled ? mean + bt : fmaf(g, mean, bt)) : 0.0f;
  }
  const float ss = wave_sum(mean * mean);
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  float tot = 0.0f;
#pragma unroll
  for (int w = 0; w < 16; ++w) tot += red[w];
  const float inv = 1.0f / fmaxf(sqrtf(tot), 1e-12f);
  if (c < H) out_row[c] = mean * inv;
}

// Block (b, q) sums rows q R .. q R + R - 1 of sequence b (all its rows when
// R == 0).  With partial == nullptr the block finishes the pooled row itself;
// otherwise it stores its column sums to partial[(b gridDim.y + q) H + c] for
// pool_combine_kernel.
template <typename T>
__global__ __launch_bounds__(1024) void pool_l2_kernel(const T* x, int H, const int* cu, float* out,
                                                       const float2* x_stats, const float* gamma, const float* beta,
                                                       float eps, bool gamma_scaled, int R, float* partial) {
  constexpr int EPC = Chunk<T>::EPC, CPL = kMaxCpl<T>;
  constexpr int kPoolBatch = 16 / CPL;  // rows per wave in flight
  extern __shared__ float part[];  // [16][H]
  __shared__ float red[16];
  __shared__ float2 row_st[kMaxPoolRows];  // (mean, rstd) per row of a deferred-LayerNorm input
  const int b = blockIdx.x;
  // column threadIdx.x's gamma and beta for the finish, requested with the
  // sequence's bounds (clamped: threads past H load a copy they never use)
  float g = 1.0f, bt = 0.0f;
  if (x_stats && !partial) {
    const int cc = min((int)threadIdx.x, H - 1);
    g = gamma[cc];
    bt = beta[cc];
  }
  const int len = cu[b + 1] - cu[b];  // the sequence's rows
  const int r0 = cu[b] + (R ? (int)blockIdx.y * R : 0);
  const int L = R ? max(0, min(R, len - (int)blockIdx.y * R)) : len;  // this block's rows
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nch = H / EPC;
  float acc[CPL][EPC];
#pragma unroll
  for (int i = 0; i < CPL; ++i)
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[i][e] = 0.0f;
  uint4 raw[kPoolBatch][CPL];  // 16-byte chunks as loaded
  auto load_batch = [&](int rb) {
#pragma unroll
    for (int k = 0; k < kPoolBatch; ++k) {
      const T* row = x + (size_t)(r0 + min(rb + 16 * k, L - 1)) * H;  // rows past the end: loaded, not added
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        const int ch = lane + 64 * i;
        if (ch < nch) raw[k][i] = *reinterpret_cast<const uint4*>(row + ch * EPC);
      }
    }
  };
  if (wave < L) load_batch(wave);
  if (x_stats) {
    for (int r = threadIdx.x; r < L; r += 1024) row_st[r] = row_ln_stats(x_stats + (size_t)(r0 + r) * (H >> 6), H >> 6, eps);
    __syncthreads();
  }
  // a gamma-scaled row holds gamma * a: (r - mean * gamma) * rstd = gamma * LN's centred, scaled a
  float gsc[CPL][EPC];
#pragma unroll
  for (int i = 0; i < CPL; ++i)
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
      const int c = min(lane + 64 * i, nch - 1) * EPC + e;
      gsc[i][e] = gamma_scaled ? gamma[c] : 1.0f;
    }
  for (int rb = wave; rb < L; rb += 16 * kPoolBatch) {
    if (rb != wave) load_batch(rb);
#pragma unroll
    for (int k = 0; k < kPoolBatch; ++k) {
      const int r = rb + 16 * k;
      if (r >= L) break;
      // (0, 1) leaves plain rows as they are
      const float2 st = x_stats ? row_st[r] : make_float2(0.0f, 1.0f);
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        const int ch = lane + 64 * i;
        if (ch < nch) {
          float v[EPC];
          Chunk<T>::from_raw(raw[k][i], v);
#pragma unroll
          for (int e = 0; e < EPC; ++e) acc[i][e] += fmaf(-st.x, gsc[i][e], v[e]) * st.y;
        }
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
  const int c = threadIdx.x;
  float sum = 0.0f;
  if (c < H) {
#pragma unroll
    for (int w = 0; w < 16; ++w) sum += part[w * H + c];
  }
  if (partial) {
    if (c < H) partial[((size_t)b * gridDim.y + blockIdx.y) * H + c] = sum;
    return;
  }
  pool_finish(sum, len, H, x_stats != nullptr, gamma_scaled, g, bt, out + (size_t)b * H, red);
}

// Adds the Q partial column sums of sequence b (in block order, so the
// result does not depend on timing) and finishes the pooled row.
__global__ __launch_bounds__(1024) void pool_combine_kernel(const float* partial, int Q, int H, const int* cu,
                                                            float* out, bool deferred, const float* gamma,
                                                            const float* beta, bool gamma_scaled) {
  __shared__ float red[16];
  const int b = blockIdx.x, c = threadIdx.x;
  float g = 1.0f, bt = 0.0f;
  if (deferred) {
    const int cc = min(c, H - 1);
    g = gamma[cc];
    bt = beta[cc];
  }
  float sum = 0.0f;
  if (c < H)
    for (int q = 0; q < Q; ++q) sum += partial[((size_t)b * Q + q) * H + c];
  pool_finish(sum, cu[b + 1] - cu[b], H, deferred, gamma_scaled, g, bt, out + (size_t)b * H, red);
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
// 16-byte chunks per lane that a row of H elements needs (H <= 1024): 1, 2 or 4
template <typename T> inline int row_chunks(int H) {
  const int per = 64 * Chunk<T>::EPC;  // elements one chunk per lane covers
  return H <= per ? 1 : H <= 2 * per ? 2 : 4;
}

}  // namespace

hipError_t launch_mask_scan(const uint8_t* mask, int B, int S, int* cu, int* tok_src, int* tok_dst, int* order,
                            hipStream_t s, int2* rank_rows) {
  if (B < 1 || S < 1 || S > 64 * kScanMaxChunks) return hipErrorInvalidValue;
  const int nch = S <= 64 ? 1 : S <= 128 ? 2 : S <= 256 ? 4 : 8;
  int* ord = B <= kMaxOrderedBatch ? order : nullptr;
  int2* rr = ord ? rank_rows : nullptr;
  // counts / prefix [B+1], then the ranks [B] only when the order is written
  // (B <= 8192 sequences stay within the default 64 KB of dynamic LDS)
  const size_t lds = (size_t)(B + 1 + (ord ? B : 0)) * sizeof(int);
  RLX_LOG_LAUNCH("mask_scan_kernel", dim3(1), dim3(1024), lds, "B=%d S=%d chunks=%d", B, S, nch);
  switch (nch) {
    case 1: hipLaunchKernelGGL(mask_scan_kernel<1>, dim3(1), dim3(1024), lds, s, mask, B, S, cu, tok_src, tok_dst, ord, rr); break;
    case 2: hipLaunchKernelGGL(mask_scan_kernel<2>, dim3(1), dim3(1024), lds, s, mask, B, S, cu, tok_src, tok_dst, ord, rr); break;
    case 4: hipLaunchKernelGGL(mask_scan_kernel<4>, dim3(1), dim3(1024), lds, s, mask, B, S, cu, tok_src, tok_dst, ord, rr); break;
    default: hipLaunchKernelGGL(mask_scan_kernel<8>, dim3(1), dim3(1024), lds, s, mask, B, S, cu, tok_src, tok_dst, ord, rr); break;
  }
  return hipGetLastError();
}

hipError_t launch_embed_ln(const int* ids, const void* word, const void* pos, const void* type, const float* gamma,
                           const float* beta, float eps, int vocab, int S, int H, const int* tok_src,
                           const int* n_dev, int n_max, void* x, DType dt, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  RLX_LOG_LAUNCH("embed_ln_kernel", dim3(blocks_for_rows(n_max)), dim3(256), 0, "%s rows<=%d H=%d", dt == DType::BF16 ? "bf16" : "f32", n_max, H);
  const dim3 grid(blocks_for_rows(n_max));
#define RLX_EMBED_LN(TT, NC)                                                                                 \
  hipLaunchKernelGGL((embed_ln_kernel<TT, NC>), grid, dim3(256), 0, s, ids, (const TT*)word, (const TT*)pos,    \
                     (const TT*)type, gamma, beta, eps, vocab, S, H, tok_src, n_dev, n_max, (TT*)x)
  switch (dt == DType::BF16 ? 10 + row_chunks<bf16_t>(H) : row_chunks<float>(H)) {
    case 11: RLX_EMBED_LN(bf16_t, 1); break;
    case 12: RLX_EMBED_LN(bf16_t, 2); break;
    case 1: RLX_EMBED_LN(float, 1); break;
    case 2: RLX_EMBED_LN(float, 2); break;
    default: RLX_EMBED_LN(float, 4); break;
  }
#undef RLX_EMBED_LN
  return hipGetLastError();
}

hipError_t launch_embed_scan(const uint8_t* mask, const int* ids, int B, int S, const void* word, const void* pos,
                             const void* type, const float* gamma, const float* beta, float eps, int vocab, int H,
                             int* cu, int* tok_src, int* tok_dst, int* order, void* x, DType dt, hipStream_t s,
                             int2* rank_rows) {
  if (B <= 0 || S <= 0) return hipSuccess;
  if (!embed_scan_supported(B, S)) return hipErrorInvalidValue;
  if (!order) rank_rows = nullptr;  // (the table follows the order)
  const dim3 grid(B, (S + kEmbedScanTokens - 1) / kEmbedScanTokens);
  RLX_LOG_LAUNCH("embed_scan_kernel", grid, dim3(256), 0, "mask scan + embedding %s B=%d S=%d H=%d", dt == DType::BF16 ? "bf16" : "f32", B, S, H);
  // chunks of 16 bytes per lane that a row needs: bf16 1 (H <= 512) or 2, f32 2 (H <= 512) or 4
  if (dt == DType::BF16) {
    if (H <= 64 * Chunk<bf16_t>::EPC)
      hipLaunchKernelGGL((embed_scan_kernel<bf16_t, 1>), grid, dim3(256), 0, s, mask, ids, B, S, (const bf16_t*)word,
                         (const bf16_t*)pos, (const bf16_t*)type, gamma, beta, eps, vocab, H, cu, tok_src, tok_dst,
                         order, (bf16_t*)x, rank_rows);
    else
      hipLaunchKernelGGL((embed_scan_kernel<bf16_t, 2>), grid, dim3(256), 0, s, mask, ids, B, S, (const bf16_t*)word,
                         (const bf16_t*)pos, (const bf16_t*)type, gamma, beta, eps, vocab, H, cu, tok_src, tok_dst,
                         order, (bf16_t*)x, rank_rows);
  } else {
    if (H <= 128 * Chunk<float>::EPC)
      hipLaunchKernelGGL((embed_scan_kernel<float, 2>), grid, dim3(256), 0, s, mask, ids, B, S, (const float*)word,
                         (const float*)pos, (const float*)type, gamma, beta, eps, vocab, H, cu, tok_src, tok_dst,
                         order, (float*)x, rank_rows);
    else
      hipLaunchKernelGGL((embed_scan_kernel<float, 4>), grid, dim3(256), 0, s, mask, ids, B, S, (const float*)word,
                         (const float*)pos, (const float*)type, gamma, beta, eps, vocab, H, cu, tok_src, tok_dst,
                         order, (float*)x, rank_rows);
  }
  return hipGetLastError();
}

hipError_t launch_gather_rows(const void* hidden, int H, const int* tok_src, const int* n_dev, int n_max, void* x,
                              DType dt, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  RLX_LOG_LAUNCH("gather_rows_kernel", dim3(blocks_for_rows(n_max)), dim3(256), 0, "%s rows<=%d H=%d", dt == DType::BF16 ? "bf16" : "f32", n_max, H);
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
  RLX_LOG_LAUNCH("layer_norm_kernel", dim3(blocks_for_rows(n_max)), dim3(256), 0, "%s rows<=%d H=%d", dt == DType::BF16 ? "bf16" : "f32", n_max, H);
  const dim3 grid(blocks_for_rows(n_max));
  switch (dt == DType::BF16 ? 10 + row_chunks<bf16_t>(H) : row_chunks<float>(H)) {
    case 11:
      hipLaunchKernelGGL((layer_norm_kernel<bf16_t, 1>), grid, dim3(256), 0, s, (const bf16_t*)a, gamma, beta, eps, H,
                         n_dev, n_max, (bf16_t*)y);
      break;
    case 12:
      hipLaunchKernelGGL((layer_norm_kernel<bf16_t, 2>), grid, dim3(256), 0, s, (const bf16_t*)a, gamma, beta, eps, H,
                         n_dev, n_max, (bf16_t*)y);
      break;
    case 1:
      hipLaunchKernelGGL((layer_norm_kernel<float, 1>), grid, dim3(256), 0, s, (const float*)a, gamma, beta, eps, H,
                         n_dev, n_max, (float*)y);
      break;
    case 2:
      hipLaunchKernelGGL((layer_norm_kernel<float, 2>), grid, dim3(256), 0, s, (const float*)a, gamma, beta, eps, H,
                         n_dev, n_max, (float*)y);
      break;
    default:
      hipLaunchKernelGGL((layer_norm_kernel<float, 4>), grid, dim3(256), 0, s, (const float*)a, gamma, beta, eps, H,
                         n_dev, n_max, (float*)y);
      break;
  }
  return hipGetLastError();
}

hipError_t launch_pool_l2(const void* x, int H, const int* cu, int B, float* out, DType dt, hipStream_t s,
                          const float2* x_stats, const float* gamma, const float* beta, float eps, bool gamma_scaled,
                          int S, float* scratch, size_t scratch_bytes) {
  if (B <= 0) return hipSuccess;
  if (gamma_scaled && !x_stats) return hipErrorInvalidValue;
  if (dt != DType::BF16 && x_stats) return hipErrorInvalidValue;
  if (H > 1024 || S > kMaxPoolRows) return hipErrorInvalidValue;
  const size_t lds = (size_t)16 * H * sizeof(float);
  // Sequences of up to S > kPoolSplitAbove rows are summed by
  // ceil(S / kPoolSplitRows) blocks each, then combined, when the scratch
  // holds the partial sums (one block per sequence takes about as long as the
  // second launch up to 128 rows, whose loads are all in flight at once).
  const int Q = (S + kPoolSplitRows - 1) / kPoolSplitRows;
  const bool split = S > kPoolSplitAbove && scratch && (size_t)B * Q * H * sizeof(float) <= scratch_bytes;
  const dim3 grid(B, split ? Q : 1);
  const int R = split ? kPoolSplitRows : 0;
  float* partial = split ? scratch : nullptr;
  RLX_LOG_LAUNCH("pool_l2_kernel", grid, dim3(1024), lds, "%s B=%d H=%d%s%s", dt == DType::BF16 ? "bf16" : "f32", B, H,
                 x_stats ? (gamma_scaled ? " deferred-LN input (gamma-scaled)" : " deferred-LN input") : "",
                 split ? " partial sums" : "");
  if (dt == DType::BF16)
    hipLaunchKernelGGL(pool_l2_kernel<bf16_t>, grid, dim3(1024), lds, s, (const bf16_t*)x, H, cu, out, x_stats,
                       gamma, beta, eps, gamma_scaled, R, partial);
  else
    hipLaunchKernelGGL(pool_l2_kernel<float>, grid, dim3(1024), lds, s, (const float*)x, H, cu, out, nullptr,
                       nullptr, nullptr, 0.0f, false, R, partial);
  if (!split) return hipGetLastError();
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  RLX_LOG_LAUNCH("pool_combine_kernel", dim3(B), dim3(1024), 0, "B=%d H=%d partial sums per sequence=%d", B, H, Q);
  hipLaunchKernelGGL(pool_combine_kernel, dim3(B), dim3(1024), 0, s, partial, Q, H, cu, out, x_stats != nullptr,
                     gamma, beta, gamma_scaled);
  return hipGetLastError();
}

hipError_t launch_scatter_hidden(const void* x, int H, const int* tok_dst, int n_tok, float* out, DType dt,
                                 hipStream_t s) {
  if (n_tok <= 0) return hipSuccess;
  RLX_LOG_LAUNCH("scatter_hidden_kernel", dim3(blocks_for_rows(n_tok)), dim3(256), 0, "%s positions=%d H=%d", dt == DType::BF16 ? "bf16" : "f32", n_tok, H);
  if (dt == DType::BF16)
    hipLaunchKernelGGL(scatter_hidden_kernel<bf16_t>, dim3(blocks_for_rows(n_tok)), dim3(256), 0, s,
                       (const bf16_t*)x, H, tok_dst, n_tok, out);
  else
    hipLaunchKernelGGL(scatter_hidden_kernel<float>, dim3(blocks_for_rows(n_tok)), dim3(256), 0, s, (const float*)x, H,
                       tok_dst, n_tok, out);
  return hipGetLastError();
}

}  // namespace rlx
