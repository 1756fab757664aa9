// Block-scaled minifloat matmul on the gfx950 MX matrix cores.
//
// The paper's ScaledMatMul path (Section VI, quantized inference) multiplies
// block-scaled minifloats -- FP8 / FP6 / FP4 grids -- and checks the result
// bit for bit against an F32 reference.  The element formats are the OCP MX
// ones (E4M3, E5M2, E2M3, E3M2, E2M1, 32 elements per E8M0 scale), which is
// exactly what v_mfma_scale_f32_32x32x64_f8f6f4 consumes: the matrix core
// applies the two blocks' scales itself, so codes and scales go from memory to
// the instruction untouched and the products are exact; only the fp32
// accumulation rounds.
//
//   y[m, n] = sum_k X(m, k) W(n, k),  X(m, k) = xs[m][k/32] * code_x[m][k], likewise W
//
// Storage (one row per m or n, K along the row): FP8 one byte per code, FP6
// four codes per three bytes (little-endian bit stream), FP4 two per byte
// (lower k in the low nibble); scales [rows][K/32] bytes.
//
// Design (512 threads = 8 waves in a 4 x 2 grid, tile 256 x 128, each wave
// 64 x 64 = 2 x 2 instructions):
//  * A stage is 128 k: the rows' 128 / 96 / 64 bytes (FP8 / FP6 / FP4) go
//    global -> LDS by DMA into a 128-byte row pitch with the 16-byte chunks
//    XOR-swizzled by (row / 2) mod 8; the rows' four scale bytes per stage go
//    by a dword DMA.  Three stages (150 KB, one block per CU): two stages are
//    in flight while one is multiplied, which is what hides the memory
//    latency -- with two 128 x 128 stages per block and two blocks per CU
//    only one stage per block was in flight and every stage waited for it.
//    The tall tile keeps the tile count at or below the CU count at the
//    benchmark shape (71 x 3 tiles for M = 18048, N = 384), so no CU runs a
//    second tile after the others have finished.
//  * Operand layout of the instruction (lane l: row l % 32, half h = l / 32),
//    checked on the GPU against the oracle: FP6 / FP4 lanes hold the 32 codes
//    of block h contiguously; FP8 lanes hold bytes 16h .. 16h+15 of block 0 in
//    their first four registers and of block 1 in the last four.  Lane half h
//    supplies the scale of block h (byte 0 of the scale register).
//  * The weight rows are the instruction's A operand, the activation rows its
//    B operand, so each lane ends up with one output row and four consecutive
//    output columns per register quad: 16-byte stores.
#include "common.hpp"
#include "kernels.hpp"

namespace rlx {
namespace {

constexpr int kMxBM = 256, kMxBN = 128;
constexpr int kMxWaves = 8;
constexpr int kMxStageK = 128;     // k per stage
constexpr int kMxPitch = 128;      // LDS bytes per staged row
constexpr int kMxStages = 3;
constexpr int kMxOpBytes = (kMxBM + kMxBN) * kMxPitch;
// one 256-byte scale DMA per wave and stage: x rows, then w rows, then (the
// waves left over) a copy that is never read, so every wave issues as many
// loads per stage
constexpr int kMxScaleBytes = kMxWaves * 256;
constexpr int kMxStageBytes = kMxOpBytes + kMxScaleBytes;
// per wave per stage: (BM + BN) rows * 128 B / (8 waves * 1 KB) chunk DMAs + 1 scale DMA
constexpr int kMxLps = (kMxBM + kMxBN) * kMxPitch / (kMxWaves * 1024) + 1;
static_assert((kMxBM + kMxBN) * 4 <= kMxScaleBytes && kMxBM % 64 == 0 && kMxBN % 64 == 0, "scale DMA layout");
static_assert(kMxStages * kMxStageBytes <= 160 * 1024, "LDS");

__host__ __device__ constexpr int mx_bits(int fmt) { return fmt <= 1 ? 8 : (fmt <= 3 ? 6 : 4); }

__device__ __forceinline__ int mx_swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

typedef int mx_v8i __attribute__((ext_vector_type(8)));

// The instruction operand of one lane: row r of a staged operand, MFMA step s
// (0 or 1) of the stage, lane half h.
template <int FMT>
__device__ __forceinline__ mx_v8i mx_fragment(const uint8_t* rows, int r, int s, int h) {
  const uint8_t* base = rows + r * kMxPitch;
  auto chunk = [&](int c) { return *reinterpret_cast<const uint4*>(base + mx_swz(r, c) * 16); };
  mx_v8i v;
  if constexpr (mx_bits(FMT) == 8) {
    const uint4 a = chunk(4 * s + h), b = chunk(4 * s + 2 + h);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  } else if constexpr (mx_bits(FMT) == 6) {
    // block 2s + h is bytes 24(2s + h) .. +23: chunks (3s, 3s+1) from byte 0
    // for h = 0, chunks (3s+1, 3s+2) from byte 8 for h = 1
    const uint4 a = chunk(3 * s + h), b = chunk(3 * s + 1 + h);
    v[0] = h ? a.z : a.x; v[1] = h ? a.w : a.y; v[2] = h ? b.x : a.z;
    v[3] = h ? b.y : a.w; v[4] = h ? b.z : b.x; v[5] = h ? b.w : b.y;
    v[6] = 0; v[7] = 0;
  } else {
    const uint4 a = chunk(2 * s + h);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = 0; v[5] = 0; v[6] = 0; v[7] = 0;
  }
  return v;
}

template <int FX, int FW>
__global__ __launch_bounds__(kMxWaves * 64) void mx_gemm_kernel(MxGemmParams p) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kMxStages * kMxStageBytes];
  const int M = p.M, N = p.N, K = p.K;
  const int n_tiles = N / kMxBN;
  const int live = n_tiles * ((M + kMxBM - 1) / kMxBM);
  const int bid = blockIdx.x;
  if (bid >= live) return;
  // XCD-aware order: workgroups go round-robin over the 8 XCDs; XCD x takes a
  // contiguous run of tiles (row-major over (row tile, column tile))
  const int q8 = live >> 3, r8 = live & 7, xcd = bid & 7;
  const int tile = xcd * q8 + min(xcd, r8) + (bid >> 3);
  const int m0 = (tile / n_tiles) * kMxBM, n0 = (tile % n_tiles) * kMxBN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, l32 = lane & 31, h = lane >> 5;  // 4 x 2 waves of 64 x 64
  const int KT = K / kMxStageK;
  constexpr int RBX = kMxStageK * mx_bits(FX) / 8, RBW = kMxStageK * mx_bits(FW) / 8;  // bytes per stage row
  const size_t pitch_x = (size_t)K * mx_bits(FX) / 8, pitch_w = (size_t)K * mx_bits(FW) / 8;
  const int sb_row = K / 32;  // scale bytes per row

  // Chunk DMA: instruction i of wave w fills staged rows 8(w + 8i) .. +7; lane
  // lands at row (lane >> 3), physical chunk (lane & 7).  Chunks past the
  // format's row bytes are never read; their lanes fetch chunk 0 again.
  constexpr int CL = kMxLps - 1;
  const uint8_t* src[CL];
  int step_bytes[CL];
#pragma unroll
  for (int i = 0; i < CL; ++i) {
    const int row = (wave + kMxWaves * i) * 8 + (lane >> 3);
    const int c = mx_swz(row, lane & 7);
    if (row < kMxBM) {
      const int m = min(m0 + row, M - 1);
      src[i] = reinterpret_cast<const uint8_t*>(p.x) + (size_t)m * pitch_x + (c * 16 < RBX ? c * 16 : 0);
      step_bytes[i] = RBX;
    } else {
      src[i] = reinterpret_cast<const uint8_t*>(p.w) + (size_t)(n0 + row - kMxBM) * pitch_w + (c * 16 < RBW ? c * 16 : 0);
      step_bytes[i] = RBW;
    }
  }
  // Scale DMA, one dword per row and stage: waves 0-3 -> x rows 64w .. 64w+63,
  // waves 4-5 -> w rows 64(w-4) .. +63, waves 6-7 -> w rows again (unread)
  const uint8_t* ssrc;
  {
    constexpr int XW = kMxBM / 64, WW = kMxBN / 64;
    const int row = (wave < XW ? wave : (wave - XW) % WW) * 64 + lane;
    ssrc = wave < XW ? p.x_scales + (size_t)min(m0 + row, M - 1) * sb_row
                     : p.w_scales + (size_t)(n0 + row) * sb_row;
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)smem;
  auto issue = [&](int kt, int buf) {
    const uint32_t sbase = lds0 + buf * kMxStageBytes;
#pragma unroll
    for (int i = 0; i < CL; ++i)
      lds_dma16(src[i] + (size_t)kt * step_bytes[i],
                __builtin_amdgcn_readfirstlane(sbase + (wave + kMxWaves * i) * 8 * kMxPitch));
    lds_dma4(ssrc + kt * 4, __builtin_amdgcn_readfirstlane(sbase + kMxOpBytes + wave * 256));
  };

  typedef float f32x16 __attribute__((ext_vector_type(16)));
  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;

  // Stages kt and kt + 1 are in flight when stage kt's wait begins; stage
  // kt + 2 is issued after the barrier that follows it, into the buffer of
  // stage kt - 1, which every wave has finished multiplying by then.
  static_assert(kMxStages == 3, "the ring below keeps two stages ahead");
  issue(0, 0);
  if (KT > 1) issue(1, 1);
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt % kMxStages;
    if (kt + 1 < KT)
      wait_vmcnt<kMxLps>();  // stage kt landed; kt + 1 in flight
    else
      wait_vmcnt<0>();
    __syncthreads();
    if (kt + 2 < KT) issue(kt + 2, (kt + 2) % kMxStages);
    const uint8_t* xs = smem + buf * kMxStageBytes;
    const uint8_t* ws = xs + kMxBM * kMxPitch;
    const uint32_t* sx = reinterpret_cast<const uint32_t*>(xs + kMxOpBytes);  // [BM] x rows, then [BN] w rows
    const uint32_t* sw = sx + kMxBM;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      mx_v8i xf[2], wf[2];
      int xsc[2], wsc[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int rx = wm * 64 + t * 32 + l32, rw = wn * 64 + t * 32 + l32;
        xf[t] = mx_fragment<FX>(xs, rx, s, h);
        wf[t] = mx_fragment<FW>(ws, rw, s, h);
        xsc[t] = (int)((sx[rx] >> (8 * (2 * s + h))) & 0xFF);
        wsc[t] = (int)((sw[rw] >> (8 * (2 * s + h))) & 0xFF);
      }
#pragma unroll
      for (int tm = 0; tm < 2; ++tm)
#pragma unroll
        for (int tn = 0; tn < 2; ++tn)
          acc[tm][tn] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(wf[tn], xf[tm], acc[tm][tn], FW, FX, 0,
                                                                         wsc[tn], 0, xsc[tm]);
    }
  }

  // Epilogue through LDS (the stage ring is free once every wave is past the
  // loop): lane holds output row wm*64 + tm*32 + l32 of the tile and, per
  // register quad i, columns wn*64 + tn*32 + 8i + 4h .. +3.  The tile goes to
  // LDS row-major, then every wave stores whole 512-byte rows: written from
  // the instruction layout, each store touched 32 rows with 32 bytes apiece.
  constexpr int kOutPitch = kMxBN + 4;  // floats per LDS row (16-byte aligned, rows 4 banks apart)
  static_assert(kMxBM * kOutPitch * 4 <= kMxStages * kMxStageBytes, "output tile in the stage ring");
  float* out_lds = reinterpret_cast<float*>(smem);
  __syncthreads();
#pragma unroll
  for (int tm = 0; tm < 2; ++tm)
#pragma unroll
    for (int tn = 0; tn < 2; ++tn)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wm * 64 + tm * 32 + l32, c = wn * 64 + tn * 32 + 8 * i + 4 * h;
        *reinterpret_cast<float4*>(out_lds + r * kOutPitch + c) =
            make_float4(acc[tm][tn][4 * i], acc[tm][tn][4 * i + 1], acc[tm][tn][4 * i + 2], acc[tm][tn][4 * i + 3]);
      }
  __syncthreads();
  constexpr int kRowThreads = kMxBN / 4;                       // float4 per row
  constexpr int kRowsPerPass = kMxWaves * 64 / kRowThreads;    // rows stored per pass
  const int rr = tid / kRowThreads, c4 = (tid % kRowThreads) * 4;
#pragma unroll 4
  for (int r = rr; r < kMxBM; r += kRowsPerPass) {
    const int m = m0 + r;
    if (m < M)
      *reinterpret_cast<float4*>(p.y + (size_t)m * N + n0 + c4) = *reinterpret_cast<const float4*>(out_lds + r * kOutPitch + c4);
  }
}

template <int FX, int FW>
hipError_t launch_mx_typed(const MxGemmParams& p, hipStream_t s) {
  const int tiles = (p.N / kMxBN) * ((p.M + kMxBM - 1) / kMxBM);
  RLX_LOG_LAUNCH("mx_gemm_kernel", dim3(tiles), dim3(kMxWaves * 64), 0, "formats=%d,%d M=%d N=%d K=%d", (int)FX,
                 (int)FW, p.M, p.N, p.K);
  hipLaunchKernelGGL((mx_gemm_kernel<FX, FW>), dim3(tiles), dim3(kMxWaves * 64), 0, s, p);
  return hipGetLastError();
}

template <int FX>
hipError_t launch_mx_w(const MxGemmParams& p, hipStream_t s) {
  switch (p.fw) {
    case 0: return launch_mx_typed<FX, 0>(p, s);
    case 1: return launch_mx_typed<FX, 1>(p, s);
    case 2: return launch_mx_typed<FX, 2>(p, s);
    case 3: return launch_mx_typed<FX, 3>(p, s);
    case 4: return launch_mx_typed<FX, 4>(p, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

bool mx_gemm_supported(int M, int N, int K) { return M >= 0 && N > 0 && K > 0 && N % 128 == 0 && K % 128 == 0; }

hipError_t launch_mx_gemm(const MxGemmParams& p, hipStream_t s) {
  if (!mx_gemm_supported(p.M, p.N, p.K) || p.fx < 0 || p.fx > 4 || p.fw < 0 || p.fw > 4) return hipErrorInvalidValue;
  if (p.M == 0) return hipSuccess;
  switch (p.fx) {
    case 0: return launch_mx_w<0>(p, s);
    case 1: return launch_mx_w<1>(p, s);
    case 2: return launch_mx_w<2>(p, s);
    case 3: return launch_mx_w<3>(p, s);
    case 4: return launch_mx_w<4>(p, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace rlx
