// Fused masked multi-head attention for gfx950.
//
// The paper's IR carries attention as one primitive parameterised by an
// explicit MaskKind in {None, Causal, SlidingWindow(w), Custom} (Section
// III-A), and its optimizer fuses the attention block and reads Q, K and V as
// strided narrows of one buffer (Section III-B).  Here that is one kernel that
// reads Q/K/V by row stride straight out of the fused QKV projection.
//
// bf16 kernel -- blocks of eight waves per (query tile of 128, head,
// sequence): four query sub-tiles of 32, each walked by two waves that take
// one half of its visible key tiles apiece and merge their softmax states
// (max, denominator, unnormalised context) through LDS at the end.  When there
// are fewer than two tiles per CU, some tiles are split into two half blocks
// (64 queries, four waves per sub-tile) so that every CU holds the same work:
//  * K rows and V (transposed) for the block's key range are staged once in
//    LDS; key tiles of 32 whose keys are all masked are skipped, and tiles
//    that every query of the sub-tile sees in full skip the mask arithmetic.
//  * Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16
//    (d = 32 is two k-steps), so each lane holds 16 keys of a single query:
//    the softmax max / sum over keys is 15 in-lane steps plus one exchange
//    with the partner lane 32 away.
//  * Online softmax in fp32 in base 2 (p = 2^(s c - m c), c = scale log2 e, as one fma),
//    the state rescaled only when some query's maximum grows), then P is
//    rounded to bf16 and multiplied into ctx^T = V^T P^T,
//    again on the matrix cores.  The probabilities stay in registers: their
//    C-layout is used directly as the B operand, with the V^T operand read in
//    the matching (permuted) key order.
//  * Two layouts: padded (rows b*S .. b*S+S-1, optional u8 key mask) and
//    variable-length (rows cu[b] .. cu[b+1]-1, every row a real token), which
//    the encoder uses after compacting away padded tokens.
// fp32 kernel -- one thread per query, K/V staged in LDS, scalar online softmax.
#include <math.h>

#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"
#include "qkv_attention.hpp"

namespace rlx {
namespace {

constexpr int kQBlock = 128;
constexpr int kKRow = 80;  // bytes per staged K row (64 + 16 pad)
constexpr float kLog2e = 1.4426950408889634f;

struct SeqRange {
  int row0, n;
};

__device__ __forceinline__ SeqRange seq_range(const AttnParams& p, int b) {
  if (p.cu_seqlens) {
    int r0 = p.cu_seqlens[b];
    return {r0, p.cu_seqlens[b + 1] - r0};
  }
  return {b * p.S, p.S};
}

// Key range [lo, hi) that queries [q_begin, q_end) may see, before the key mask.
__device__ __forceinline__ void key_bounds(const AttnParams& p, int n, int q_begin, int q_end, int& lo, int& hi) {
  lo = 0;
  hi = n;
  if (p.kind == 1 || p.kind == 2) hi = min(n, q_end);
  if (p.kind == 2) lo = max(0, q_begin - p.window + 1);
}

__device__ __forceinline__ bool visible(int kind, int window, int qi, int key) {
  if (kind == 1) return key <= qi;
  if (kind == 2) return key <= qi && key > qi - window;
  return true;
}

// Whole 32-key tile [key0, key0 + 32) visible to every query of [q0, q0 + 32)
// under the positional part of the mask (the key mask is checked separately).
__device__ __forceinline__ bool tile_fully_visible(int kind, int window, int q0, int key0) {
  if (kind == 1) return key0 + 31 <= q0;
  if (kind == 2) return key0 + 31 <= q0 && key0 > q0 + 31 - window;
  return true;
}

// Partial softmax states of the waves that hand theirs to a sub-tile's first
// wave through LDS: [query sub-tile][key part - 1][m, l, acc[16]][lane]
// (4 sub-tiles x 1 part, or 2 sub-tiles x 3 parts).
constexpr int kPartFloats = 18;
constexpr size_t kPartBytes = (size_t)6 * kPartFloats * 64 * 4;

// Blocks of eight waves.  A whole block takes a query tile of 128: four
// sub-tiles of 32, each walked by two waves that split its key tiles.  A half
// block takes 64 queries of a tile: two sub-tiles, each split over four waves.
// Block -> work: workgroups go to the eight XCDs round-robin (block i to XCD
// i % 8), and each XCD is given a contiguous run of query tiles (tile index
// fastest, the tile with the most visible keys first, then head, then
// sequence), so the tiles of one (head, sequence) share one L2.  With
// nfull >= 0 the first nfull / 8 tiles of each XCD's run are whole blocks and
// the rest are split into two half blocks; with nfull < 0 every tile is a
// whole block and the XCD runs apply when the block count is a multiple of 8.
__global__ __launch_bounds__(512) void attn_bf16_kernel(AttnParams p, int vt_stride, int gx, int nfull) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int total = (int)gridDim.x;
  int lin, qhalf = -1;  // query tile, and which half of it (-1: the whole tile)
  if (nfull >= 0) {
    const int tq = gx * p.heads * p.B / 8, fx = nfull / 8;
    const int x = (int)blockIdx.x & 7, j = (int)blockIdx.x >> 3;
    if (j < fx) {
      lin = x * tq + j;
    } else {
      lin = x * tq + fx + ((j - fx) >> 1);
      qhalf = (j - fx) & 1;
    }
  } else {
    lin = (int)blockIdx.x;
    if ((total & 7) == 0) lin = (lin & 7) * (total >> 3) + (lin >> 3);
  }
  const int qt = gx - 1 - lin % gx;
  const int h = (lin / gx) % p.heads, b = lin / gx / p.heads;
  const SeqRange sr = seq_range(p, b);
  const int n = sr.n;
  const int q_begin = qt * kQBlock + (qhalf > 0 ? kQBlock / 2 : 0);
  if (q_begin >= n) return;
  const int q_end = min(n, q_begin + (qhalf >= 0 ? kQBlock / 2 : kQBlock));
  const int nsub = qhalf >= 0 ? 2 : 4, nsplit = 8 / nsub;  // query sub-tiles, key parts per sub-tile

  int klo, khi;
  key_bounds(p, n, q_begin, q_end, klo, khi);
  klo &= ~31;                                  // stage whole 32-key tiles
  const int nk = ((khi - klo) + 31) & ~31;     // staged keys (0..512)
  const int ntiles = nk >> 5;

  uint8_t* k_lds = smem;                                                  // [nk][80 B]
  bf16_t* vt_lds = reinterpret_cast<bf16_t*>(smem + (size_t)nk * kKRow);  // [32][vt_stride]
  uint32_t* kbits = reinterpret_cast<uint32_t*>(smem + (size_t)nk * kKRow + 32 * vt_stride * 2);

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int sub = wave & (nsub - 1), kp = wave / nsub;  // query sub-tile of 32, key part
  const bf16_t* kg = reinterpret_cast<const bf16_t*>(p.k);
  const bf16_t* vg = reinterpret_cast<const bf16_t*>(p.v);
  const bf16_t* qg = reinterpret_cast<const bf16_t*>(p.q);
  const size_t ld = (size_t)p.ld_qkv;
  const int col = h * 32;

  const int q0 = q_begin + sub * 32;
  const bool active = q0 < n;
  const int l32 = lane & 31, half = lane >> 5;
  const int qi = q0 + l32;
  const int qrow = sr.row0 + min(qi, n - 1);
  uint4 qa = *reinterpret_cast<const uint4*>(qg + (size_t)qrow * ld + col + half * 8);
  uint4 qb = *reinterpret_cast<const uint4*>(qg + (size_t)qrow * ld + col + 16 + half * 8);
  if (p.scale < 0.0f) {  // fold the sign into Q (exact) so the running max is over raw scores
    qa.x ^= 0x80008000u; qa.y ^= 0x80008000u; qa.z ^= 0x80008000u; qa.w ^= 0x80008000u;
    qb.x ^= 0x80008000u; qb.y ^= 0x80008000u; qb.z ^= 0x80008000u; qb.w ^= 0x80008000u;
  }

  // Stage K (row-major) and V (transposed): thread t takes keys 4(t/4) .. +3,
  // dimensions 8(t%4) .. +7; all eight 16-byte loads are issued before any
  // store.  Keys past the sequence are zero.
  if (tid < nk) {
    const int kq = tid >> 2, c = tid & 3;
    uint4 kv[4], vv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int key = klo + 4 * kq + j;
      kv[j] = make_uint4(0, 0, 0, 0);
      vv[j] = make_uint4(0, 0, 0, 0);
      if (key < n) {
        const size_t off = (size_t)(sr.row0 + key) * ld + col + c * 8;
        kv[j] = *reinterpret_cast<const uint4*>(kg + off);
        vv[j] = *reinterpret_cast<const uint4*>(vg + off);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) *reinterpret_cast<uint4*>(k_lds + (4 * kq + j) * kKRow + c * 16) = kv[j];
    // V^T row 8c + e, keys 4kq .. 4kq+3: one 8-byte store per dimension.
    auto word = [](const uint4& u, int w) { return w == 0 ? u.x : (w == 1 ? u.y : (w == 2 ? u.z : u.w)); };
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t a0 = word(vv[0], w), a1 = word(vv[1], w), a2 = word(vv[2], w), a3 = word(vv[3], w);
      bf16_t* dst = vt_lds + (size_t)(c * 8 + 2 * w) * vt_stride + 4 * kq;
      *reinterpret_cast<uint2*>(dst) = make_uint2((a0 & 0xffffu) | (a1 << 16), (a2 & 0xffffu) | (a3 << 16));
      *reinterpret_cast<uint2*>(dst + vt_stride) = make_uint2((a0 >> 16) | (a1 & 0xffff0000u),
                                                                 (a2 >> 16) | (a3 & 0xffff0000u));
    }
  }
  // Per-tile validity bits (key inside the sequence and allowed by the key mask).
  for (int t = wave; t < ntiles; t += 8) {
    const int key = klo + t * 32 + (lane & 31);
    bool ok = key < n;
    if (ok && p.key_mask) ok = p.key_mask[(size_t)b * p.S + key] != 0;
    const uint64_t bal = __ballot(ok && lane < 32);
    if (lane == 0) kbits[t] = (uint32_t)bal;
  }
  __syncthreads();

  const bf16x8_t qf0 = as_bf16x8(qa), qf1 = as_bf16x8(qb);
  // The sub-tile's tiles holding a visible key, split between its waves in
  // key order: part k takes ranks [ceil(k c / P), ceil((k + 1) c / P)) of the
  // c such tiles (P parts).  The split depends only on those tiles, so
  // appending masked keys to a sequence leaves every result bit-identical.
  int t_begin = 0, t_end = 0;
  if (active) {
    int wlo, whi;
    key_bounds(p, n, q0, min(n, q0 + 32), wlo, whi);
    const int a = max(0, (wlo - klo) >> 5), e = min(ntiles, (whi - klo + 31) >> 5);
    int live = 0;
    for (int t = a; t < e; ++t) live += kbits[t] != 0u;
    const int r0 = (kp * live + nsplit - 1) / nsplit, r1 = ((kp + 1) * live + nsplit - 1) / nsplit;
    t_begin = e;
    t_end = e;
    for (int t = a, c = 0; t < e; ++t) {
      if (kbits[t] == 0u) continue;
      if (c == r0) t_begin = t;
      if (c == r1) {
        t_end = t;
        break;
      }
      ++c;
    }
    t_begin = min(t_begin, t_end);
  }

  // Kept above zero so that masked scores (-inf) stay -inf after the scaling.
  const float sl2 = fmaxf(fabsf(p.scale) * kLog2e, 1e-30f);
  const int xor32 = (lane ^ 32) << 2;  // ds_bpermute address of the partner lane
  float m_run = -INFINITY;  // running max of the raw scores of this query (both lanes agree)
  float l_run = 0.0f;       // this lane's share of the running denominator, relative to m_run
  f32x16_t acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.0f;

  for (int t = t_begin; t < t_end; ++t) {
    const uint32_t bits = __builtin_amdgcn_readfirstlane(kbits[t]);
    if (bits == 0u) continue;
    const int kb = t * 32;
    const uint8_t* krow = k_lds + (kb + l32) * kKRow + half * 16;
    f32x16_t s;
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = 0.0f;
    s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(*reinterpret_cast<const uint4*>(krow)), qf0, s, 0, 0, 0);
    s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(*reinterpret_cast<const uint4*>(krow + 32)), qf1, s, 0, 0,
                                                0);
    // Register v holds key kb + 8*(v/4) + 4*half + (v%4) for query qi.
    float tmax = -INFINITY;
    if (bits == 0xffffffffu && tile_fully_visible(p.kind, p.window, q0, klo + kb)) {
#pragma unroll
      for (int v = 0; v < 16; ++v) tmax = fmaxf(tmax, s[v]);
    } else {
      // This lane's visible keys of the tile as a bit mask (bit kk = key
      // klo + kb + kk), shifted so that register v tests a constant bit.
      uint32_t vis = bits;
      if (p.kind == 1 || p.kind == 2) {
        const int rel = qi - (klo + kb);  // keys kk <= rel are not in the future
        vis &= rel >= 31 ? ~0u : (rel < 0 ? 0u : (2u << rel) - 1u);
        if (p.kind == 2) {
          const int lo = rel - p.window + 1;  // keys kk >= lo are inside the window
          vis &= lo <= 0 ? ~0u : (lo >= 32 ? 0u : ~0u << lo);
        }
      }
      vis >>= 4 * half;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        s[v] = (vis >> (8 * (v >> 2) + (v & 3))) & 1u ? s[v] : -INFINITY;
        tmax = fmaxf(tmax, s[v]);
      }
    }
    tmax = fmaxf(tmax, __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(xor32, __builtin_bit_cast(int, tmax))));
    if (__any(tmax > m_run)) {  // some query's maximum grew: rescale its state
      const float alpha = tmax > m_run ? __builtin_amdgcn_exp2f((m_run - tmax) * sl2) : 1.0f;
      l_run *= alpha;
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[v] *= alpha;
      m_run = fmaxf(m_run, tmax);
    }
    // p = exp2(sl2 * (s - m)) with the bare hardware exp2 (results below
    // 2^-126 flush to zero); a query with nothing visible yet has s = -inf
    // everywhere and gets p = 0.
    const float mb = m_run == -INFINITY ? 0.0f : m_run * sl2;
    float pv[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) pv[v] = __builtin_amdgcn_exp2f(fmaf(s[v], sl2, -mb));
    float psum = 0.0f;
#pragma unroll
    for (int v = 0; v < 16; v += 4) psum += (pv[v] + pv[v + 1]) + (pv[v + 2] + pv[v + 3]);
    l_run += psum;

    const uint4 pb0 = make_uint4(pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]), pack_bf16x2(pv[4], pv[5]),
                                 pack_bf16x2(pv[6], pv[7]));
    const uint4 pb1 = make_uint4(pack_bf16x2(pv[8], pv[9]), pack_bf16x2(pv[10], pv[11]),
                                 pack_bf16x2(pv[12], pv[13]), pack_bf16x2(pv[14], pv[15]));
    // V^T operand: row d = l32, keys kb + 4*half + {0..3} and kb + 8 + 4*half + {0..3} (+16 for step 2).
    const bf16_t* vrow = vt_lds + (size_t)l32 * vt_stride + kb + 4 * half;
    const uint2 v00 = *reinterpret_cast<const uint2*>(vrow);
    const uint2 v01 = *reinterpret_cast<const uint2*>(vrow + 8);
    const uint2 v10 = *reinterpret_cast<const uint2*>(vrow + 16);
    const uint2 v11 = *reinterpret_cast<const uint2*>(vrow + 24);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(make_uint4(v00.x, v00.y, v01.x, v01.y)),
                                                  as_bf16x8(pb0), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(make_uint4(v10.x, v10.y, v11.x, v11.y)),
                                                  as_bf16x8(pb1), acc, 0, 0, 0);
  }

  // Merge the key parts of each query sub-tile into its first wave (the K / V
  // staging area is free once every wave has passed the barrier).
  __syncthreads();
  float* part = reinterpret_cast<float*>(smem) + (size_t)sub * (nsplit - 1) * kPartFloats * 64 + lane;
  if (kp > 0 && active) {
    float* pp = part + (size_t)(kp - 1) * kPartFloats * 64;
    pp[0] = m_run;
    pp[64] = l_run;
#pragma unroll
    for (int v = 0; v < 16; ++v) pp[(2 + v) * 64] = acc[v];
  }
  __syncthreads();
  if (kp > 0 || !active) return;
  float m = m_run;
  for (int k = 1; k < nsplit; ++k) m = fmaxf(m, part[(size_t)(k - 1) * kPartFloats * 64]);
  // A part that saw no key has m = -inf and weight 0; so has every part of a
  // query with no visible key (m = -inf), whose output is then zero.
  const float a0 = m == -INFINITY ? 0.0f : exp2f((m_run - m) * sl2);
  float l_lane = a0 * l_run;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] *= a0;
  for (int k = 1; k < nsplit; ++k) {
    const float* pp = part + (size_t)(k - 1) * kPartFloats * 64;
    const float ak = m == -INFINITY ? 0.0f : exp2f((pp[0] - m) * sl2);
    l_lane += ak * pp[64];
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] += ak * pp[(2 + v) * 64];
  }
  const float l_tot = l_lane + __shfl_xor(l_lane, 32, 64);
  if (qi >= n) return;
  const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
  bf16_t* og = reinterpret_cast<bf16_t*>(p.out) + (size_t)(sr.row0 + qi) * p.ld_out + col;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int d = 8 * i + 4 * half;
    *reinterpret_cast<uint2*>(og + d) =
        make_uint2(pack_bf16x2(acc[4 * i] * inv, acc[4 * i + 1] * inv),
                   pack_bf16x2(acc[4 * i + 2] * inv, acc[4 * i + 3] * inv));
  }
}

// fp32 attention on the matrix cores (head_dim 32): a block of four waves
// takes 128 queries of one (sequence, head); wave w owns queries
// q0 + 32w .. q0 + 32w + 31.  Keys are staged into LDS 64 at a time (rows
// padded so the fragment reads are bank-conflict free, rows past the key
// range zeroed) and every wave walks the staged 32-key tiles with
//   S^T = K Q^T   16 x v_mfma_f32_32x32x2_f32  (step t contracts d = t and
//                 d = t + 16, one per lane half; Q stays in registers,
//                 pre-scaled by scale * log2 e)
//   O^T += V^T P^T 16 x v_mfma_f32_32x32x2_f32 (step s contracts the keys
//                 the two lane halves hold in score register s)
// so lane l holds query l % 32 in both products: its running max, sum and
// output rescale are lane-local, the two halves (16 keys each) combine with
// one exchange, and P goes from the score registers straight into P V.
constexpr int kF32KeyChunk = 64;
constexpr int kF32KPitch = 36;  // floats per staged K row: 16-byte reads of 16 lanes hit distinct banks
constexpr int kF32VPitch = 40;  // floats per staged V row: the two lane halves' rows are 32 banks apart

__global__ __launch_bounds__(256) void attn_f32_kernel(AttnParams p) {
  __shared__ __attribute__((aligned(16))) float k_lds[kF32KeyChunk * kF32KPitch];
  __shared__ __attribute__((aligned(16))) float v_lds[kF32KeyChunk * kF32VPitch];
  __shared__ uint8_t ok_lds[kF32KeyChunk];
  const int b = blockIdx.z, h = blockIdx.y;
  const SeqRange sr = seq_range(p, b);
  const int n = sr.n;
  const int q_begin = blockIdx.x * kQBlock;
  if (q_begin >= n) return;
  const int q_end = min(n, q_begin + kQBlock);
  int klo, khi;
  key_bounds(p, n, q_begin, q_end, klo, khi);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int qw0 = q_begin + 32 * wave;
  const bool active = qw0 < q_end;           // wave-uniform
  const int qi = min(qw0 + l32, q_end - 1);  // this lane's query (clamped for the loads)
  const float* kg = reinterpret_cast<const float*>(p.k);
  const float* vg = reinterpret_cast<const float*>(p.v);
  const float* qg = reinterpret_cast<const float*>(p.q);
  const size_t ld = (size_t)p.ld_qkv;
  const int col = h * 32;

  float qv[16];
  {
    const float sl2 = p.scale * kLog2e;
    const float4* qr = reinterpret_cast<const float4*>(qg + (size_t)(sr.row0 + qi) * ld + col + 16 * half);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float4 v = qr[i];
      qv[4 * i] = v.x * sl2; qv[4 * i + 1] = v.y * sl2; qv[4 * i + 2] = v.z * sl2; qv[4 * i + 3] = v.w * sl2;
    }
  }
  f32x16_t acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  for (int c0 = klo; c0 < khi; c0 += kF32KeyChunk) {
    // stage keys c0 .. c0 + 63: two 16-byte pieces of K and of V per thread
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int idx = tid + 256 * i, kr = idx >> 3, c = idx & 7;
      float4 kv = make_float4(0.f, 0.f, 0.f, 0.f), vv = kv;
      if (c0 + kr < khi) {
        const size_t off = (size_t)(sr.row0 + c0 + kr) * ld + col + c * 4;
        kv = *reinterpret_cast<const float4*>(kg + off);
        vv = *reinterpret_cast<const float4*>(vg + off);
      }
      *reinterpret_cast<float4*>(k_lds + kr * kF32KPitch + c * 4) = kv;
      *reinterpret_cast<float4*>(v_lds + kr * kF32VPitch + c * 4) = vv;
    }
    if (tid < kF32KeyChunk) {
      const int key = c0 + tid;
      ok_lds[tid] = key < khi && (!p.key_mask || p.key_mask[(size_t)b * p.S + key] != 0);
    }
    __syncthreads();
    if (active) {
#pragma unroll 1
      for (int t0 = 0; t0 < kF32KeyChunk; t0 += 32) {
        const int key0 = c0 + t0;
        if (key0 >= khi) break;
        // the whole tile hidden from every query of this wave by position: skip
        if ((p.kind == 1 || p.kind == 2) && key0 > min(qw0 + 31, q_end - 1)) break;
        if (p.kind == 2 && key0 + 31 <= qw0 - p.window) continue;
        // S^T tile: keys key0 + 8(r/4) + 4 half + r%4 (register r) of query qi
        f32x16_t st;
#pragma unroll
        for (int r = 0; r < 16; ++r) st[r] = 0.0f;
        const float* kr = k_lds + (t0 + l32) * kF32KPitch + 16 * half;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float4 kf = *reinterpret_cast<const float4*>(kr + 4 * i);
          st = __builtin_amdgcn_mfma_f32_32x32x2f32(kf.x, qv[4 * i], st, 0, 0, 0);
          st = __builtin_amdgcn_mfma_f32_32x32x2f32(kf.y, qv[4 * i + 1], st, 0, 0, 0);
          st = __builtin_amdgcn_mfma_f32_32x32x2f32(kf.z, qv[4 * i + 2], st, 0, 0, 0);
          st = __builtin_amdgcn_mfma_f32_32x32x2f32(kf.w, qv[4 * i + 3], st, 0, 0, 0);
        }
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kk = t0 + 8 * (r >> 2) + 4 * half + (r & 3);
          const bool vis = ok_lds[kk] && visible(p.kind, p.window, qi, c0 + kk);
          st[r] = vis ? st[r] : -INFINITY;
          mx = fmaxf(mx, st[r]);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float m_new = fmaxf(m_run, mx);
        // nothing visible to this query yet: p = 0 and alpha = 0 (acc and l
        // are still 0) with a finite reference, no divergence around the MFMAs
        const float m_ref = m_new == -INFINITY ? 0.0f : m_new;
        const float alpha = exp2f(m_run - m_ref);
        float sum = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          st[r] = exp2f(st[r] - m_ref);
          sum += st[r];
        }
        sum += __shfl_xor(sum, 32, 64);
        l_run = l_run * alpha + sum;
        m_run = m_new;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] *= alpha;
        // O^T += V^T P^T: step r takes key t0 + 8(r/4) + 4 half + r%4 in each half
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float va = v_lds[(t0 + 8 * (r >> 2) + 4 * half + (r & 3)) * kF32VPitch + l32];
          acc = __builtin_amdgcn_mfma_f32_32x32x2f32(va, st[r], acc, 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }
  // lane: query qw0 + l32, dims 8j + 4 half .. +3 in registers 4j .. 4j+3
  if (!active || qw0 + l32 >= q_end) return;
  const float inv = l_run > 0.0f ? 1.0f / l_run : 0.0f;
  float* og = reinterpret_cast<float*>(p.out) + (size_t)(sr.row0 + qw0 + l32) * p.ld_out + col + 4 * half;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    *reinterpret_cast<float4*>(og + 8 * j) =
        make_float4(acc[4 * j] * inv, acc[4 * j + 1] * inv, acc[4 * j + 2] * inv, acc[4 * j + 3] * inv);
}

}  // namespace


// ---------------------------------------------------------------------------
// QKV projection fused with attention (sequences of <= 128 tokens)
// ---------------------------------------------------------------------------
// One block per (head, sequence); the block body is qkv_attention_block
// (qkv_attention.hpp), shared with the persistent encoder forward.
namespace {

template <int STAGES>
__global__ __launch_bounds__(256) void qkv_attn_bf16_kernel(FusedAttnParams p) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[qkv_attention_ring_bytes<STAGES>()];
  __shared__ __attribute__((aligned(16))) float vec_lds[2 * kFwRows];            // this head's bias, then fold_u
  __shared__ __attribute__((aligned(16))) float2 st_lds[kFxRows * kLnMaxParts];  // [token][np] partial statistics
  // Block -> (sequence, head), XCD-aware: workgroups are dispatched
  // round-robin over the 8 XCDs (block i to XCD i % 8), and all heads of one
  // sequence are given to one XCD, so its L2 fetches the sequence's token rows
  // once instead of once per XCD.  Sequences are taken in groups of 8 by rank
  // (longest first when an order is given), one per XCD, the direction
  // alternating between groups to balance the XCDs' work.  Within an XCD the
  // items (group, head) are ranked longest first.  When an XCD has more
  // blocks than CUs but at most twice as many, its slots c and c + C (C CUs
  // per XCD) land on the same CU: all CUs are free at launch and each takes a
  // second block in the same round-robin order.  The longest items then get a
  // CU of their own, and the rest are paired longest with shortest, which
  // lowers the busiest CU's load.  Otherwise slots follow the ranks.
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int n = gridDim.x >> 3, C = p.cu_per_xcd;
  int item = slot;
  if (C > 0 && n > C && n <= 2 * C) {
    const int P = n - C;  // CUs with two blocks
    item = slot < P ? 2 * C - n + slot : (slot < C ? slot - P : n - 1 - (slot - C));
  }
  const int grp = item / p.heads, h = item - grp * p.heads;
  const int rank = 8 * grp + ((grp & 1) ? 7 - xcd : xcd);
  if (rank >= p.B) return;
  int row0, L;
  if (p.rank_rows) {  // one load: the scan wrote (first row, length) by rank
    const int2 rl = p.rank_rows[rank];
    row0 = rl.x;
    L = rl.y;
  } else {
    const int b = p.seq_order ? p.seq_order[rank] : rank;
    row0 = p.cu_seqlens[b];
    L = p.cu_seqlens[b + 1] - row0;
  }
  if (L <= 0) return;
  qkv_attention_block<STAGES>(p, row0, L, h, smem, vec_lds, st_lds, [] {});
}

}  // namespace

hipError_t launch_qkv_attention(const FusedAttnParams& p, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  RLX_LOG_LAUNCH("qkv_attn_bf16_kernel", dim3(((p.B + 7) / 8) * 8 * p.heads), dim3(256), 0,
                 "fused QKV projection + attention, stages=2 B=%d heads=%d H=%d%s", p.B, p.heads, p.H,
                 p.x_stats ? " deferred-LN input" : "");
  static const int cu_per_xcd = [] {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    return cus % 8 == 0 ? cus / 8 : 0;
  }();
  FusedAttnParams q = p;
  q.cu_per_xcd = cu_per_xcd;
  hipLaunchKernelGGL(qkv_attn_bf16_kernel<2>, dim3(((p.B + 7) / 8) * 8 * p.heads), dim3(256), 0, s, q);
  return hipGetLastError();
}

// Raise the dynamic-LDS limit of the bf16 kernel once (S = 512 needs ~74 KB;
// gfx950 has 160 KB per workgroup).  The fp32 kernel stages 64 keys at a
// time in static LDS.
hipError_t set_lds_limits() {
  static const hipError_t once = hipFuncSetAttribute(reinterpret_cast<const void*>(attn_bf16_kernel),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  return once;
}

hipError_t init_kernel_attributes() { return set_lds_limits(); }

hipError_t launch_attention(const AttnParams& p, hipStream_t s) {
  if (p.B <= 0 || p.S <= 0) return hipSuccess;
  const hipError_t le = set_lds_limits();
  if (le != hipSuccess) return le;
  const int gx = (p.S + kQBlock - 1) / kQBlock;
  if (p.dtype == DType::BF16) {
    const int nk_max = (p.S + 31) & ~31;  // staged keys never exceed the padded length
    const int vt_stride = ((nk_max + 127) & ~127) + 4;
    const size_t stage = (size_t)nk_max * kKRow + 32 * (size_t)vt_stride * 2 + (size_t)(nk_max / 32) * 4;
    const size_t lds = stage > kPartBytes ? stage : kPartBytes;
    const int64_t tiles = (int64_t)gx * p.heads * p.B;
    if (tiles > 0x3fffffff) return hipErrorInvalidValue;
    // Two blocks fit a CU.  With at most two tiles per CU, split tiles into
    // half blocks until every CU holds one whole and one half block (or two
    // halves); with fewer tiles than CUs, every tile is split.
    int cus = 0, dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return hipErrorInvalidValue;
    int nfull = -1;
    int64_t blocks = tiles;
    if (tiles % 8 == 0 && cus % 8 == 0 && tiles < 2 * (int64_t)cus) {
      nfull = (int)std::max<int64_t>(0, 2 * tiles - 2 * (int64_t)cus);
      blocks = 2 * tiles - nfull;
    }
    RLX_LOG_LAUNCH("attn_bf16_kernel", dim3((unsigned)blocks), dim3(512), lds,
                   "B=%d S=%d heads=%d kind=%d query tiles=%lld whole blocks=%d%s", p.B, p.S, p.heads, p.kind,
                   (long long)tiles, nfull < 0 ? (int)tiles : nfull, p.cu_seqlens ? " varlen" : "");
    hipLaunchKernelGGL(attn_bf16_kernel, dim3((unsigned)blocks), dim3(512), lds, s, p, vt_stride, gx, nfull);
  } else {
    const dim3 grid(gx, p.heads, p.B);
    RLX_LOG_LAUNCH("attn_f32_kernel", grid, dim3(256), 0, "B=%d S=%d heads=%d kind=%d%s", p.B, p.S, p.heads, p.kind,
                   p.cu_seqlens ? " varlen" : "");
    hipLaunchKernelGGL(attn_f32_kernel, grid, dim3(256), 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace rlx
