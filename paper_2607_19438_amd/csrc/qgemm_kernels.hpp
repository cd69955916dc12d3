// Device code of the block-quantised prefill GEMM for gfx950 (MI355X).
//
// One workgroup owns one output tile and walks the contraction dimension,
// accumulating tile products into register-resident fp32 accumulators (the
// structure Section 3.1 describes for the paper's matrix-unit kernels). On
// gfx950 the product is a bf16 MFMA (v_mfma_f32_32x32x16_bf16); the packed
// Q8 / Q4 weights are read from HBM with 16-byte loads, dequantised in
// registers (value * fp16 block scale, rounded to bf16) and staged in LDS so
// every wave of the workgroup reuses them. Activations are staged in LDS too.
// LDS is double-buffered: the single-barrier tiles (four waves, or eight waves
// side by side on 32 rows for small MoE groups) close a 64-wide K step with one
// barrier, the eight-wave ping-pong tiles with two (see tile_body).
#pragma once

#include <hip/hip_runtime.h>
#include <type_traits>
#include <stdint.h>

namespace qg {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

constexpr int kQ8 = 0;
constexpr int kQ4 = 1;
constexpr int kBK = 64;              // K elements per pipeline step (two 32-element scale blocks)
constexpr int kRowBytes = kBK * 2;   // one bf16 tile row in LDS: 128 bytes = 8 chunks of 16 bytes
constexpr int kMaxExpertsPerLaunch = 128;
// Consecutive MoE m-tile groups dealt to one XCD. Runs of 2 and 4 (an expert's neighbouring groups
// sharing an L2) measured the same launch times as 1 on the skewed T=8192 workload (gate/up 474-478
// us, down 326-333 us) and cut its gate/up fetch only from 748 to 714 / 699 MB: the groups'
// gathered activation rows, not the shared weights, fill the 4 MB L2.
constexpr int kMoeRun = 1;

// ---------------------------------------------------------------------------
// small helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));   // v_cvt_pk_bf16_f32 (RNE)
}

__device__ __forceinline__ float fp16_to_f32(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}

// Row swizzle of the 16-byte chunks of a [rows][64] bf16 LDS tile: logical chunk c of row r
// sits at slot c ^ row_swizzle(r). The map is linear over GF(2) in the low four row bits (bits
// 0..3 map to 1, 3, 5, 1; table below, one nibble per r mod 16). It keeps every access of the
// tile kernel free of bank conflicts whether a 16-byte LDS access phase serves 16 lanes over 64
// four-byte banks or 8 lanes over 32 banks:
//   fragment reads: 32 consecutive rows at one logical chunk (per lane half);
//   Q4 dequant writes: lane t writes row t / 2, chunk 4 (t % 2) + u;
//   Q8 dequant writes: lane t writes row t / 4, chunk 2 (t % 4) + u.
// (A swizzle by the row pair, (r >> 1) & 7, is conflict-free only in the first model; the
// hardware counters show the second.)
constexpr unsigned long long kRowSwizzleTable = 0x6754320176452310ull;
__host__ __device__ constexpr int row_swizzle(int r) { return (int)((kRowSwizzleTable >> (4 * (r & 15))) & 7); }

// Byte offset of 16-byte chunk `c` (0..7) of row `r` in a [rows][64] bf16 LDS tile.
__device__ __forceinline__ int lds_chunk(int r, int c) {
  return r * kRowBytes + ((c ^ row_swizzle(r)) << 4);
}

// h = silu(g) * u in fp32 (the SiLU-gated activation); shared by the fused epilogue and the
// standalone kernel so both round the same fp32 value to bf16.
// silu(g) = g / (1 + e^-g) with the hardware exponential and reciprocal (each within about one
// fp32 ulp, far below the bf16 rounding of h); g -> -inf gives 1 / inf = 0, so silu -> -0.
__device__ __forceinline__ float swiglu_f32(float g, float u) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
}

// One 16-byte LDS unit of dequantised weights = 8 bf16.
// Q8: two dwords of int8 (8 weights) with scale s.
__device__ __forceinline__ u32x4 dequant_q8_unit(uint32_t d0, uint32_t d1, float s) {
  const float f0 = (float)(int8_t)(d0), f1 = (float)(int8_t)(d0 >> 8);
  const float f2 = (float)(int8_t)(d0 >> 16), f3 = (float)(int8_t)(d0 >> 24);
  const float f4 = (float)(int8_t)(d1), f5 = (float)(int8_t)(d1 >> 8);
  const float f6 = (float)(int8_t)(d1 >> 16), f7 = (float)(int8_t)(d1 >> 24);
  return u32x4{pack_bf16x2(f0 * s, f1 * s), pack_bf16x2(f2 * s, f3 * s), pack_bf16x2(f4 * s, f5 * s),
               pack_bf16x2(f6 * s, f7 * s)};
}

// Q4: one dword of 8 nibbles (element 2b in the low nibble of byte b, 2b+1 in the high nibble).
// Each 16-bit half of (d & 0x000F000F), (d & 0x00F000F0) and the same masks of d >> 8 holds one
// nibble n (times 1 or 16) and no exponent bits, i.e. the fp16 subnormal n * 2^-24 (or
// 16 n * 2^-24). v_fma_mix_f32 widens an fp16 half exactly and computes
//   n * 2^-24 * (s * 2^24) - 8 s  =  (n - 8) * s
// with one rounding; (n - 8) * s (4 x 11 significant bits) is exact in fp32, as are s * 2^24,
// s * 2^20 and -8 s for every fp16 scale s, so the product is the exact dequantised weight and only
// the bf16 packing rounds (RNE). s24 = s * 2^24, s20 = s * 2^20, off = -8 s (all zero for a masked
// chunk). 17 VALU instructions per 8 weights (fp16 denormals are kept: float_denorm_mode_16_64).
__device__ __forceinline__ u32x4 dequant_q4_unit(uint32_t d, float s24, float s20, float off) {
  typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
  const uint32_t d8 = d >> 8;
  const f16x2 a = __builtin_bit_cast(f16x2, d & 0x000F000Fu);    // elements 0, 4
  const f16x2 b = __builtin_bit_cast(f16x2, d & 0x00F000F0u);    // elements 1, 5 (times 16)
  const f16x2 c = __builtin_bit_cast(f16x2, d8 & 0x000F000Fu);   // elements 2, 6
  const f16x2 e = __builtin_bit_cast(f16x2, d8 & 0x00F000F0u);   // elements 3, 7 (times 16)
  return u32x4{pack_bf16x2(__builtin_fmaf((float)a[0], s24, off), __builtin_fmaf((float)b[0], s20, off)),
               pack_bf16x2(__builtin_fmaf((float)c[0], s24, off), __builtin_fmaf((float)e[0], s20, off)),
               pack_bf16x2(__builtin_fmaf((float)a[1], s24, off), __builtin_fmaf((float)b[1], s20, off)),
               pack_bf16x2(__builtin_fmaf((float)c[1], s24, off), __builtin_fmaf((float)e[1], s20, off))};
}

// Q4 per-chunk factors of dequant_q4_unit from the fp16 scale s (0 for a masked chunk)
__device__ __forceinline__ void q4_factors(float s, float& s24, float& s20, float& off) {
  s24 = s * 16777216.0f;
  s20 = s * 1048576.0f;
  off = -8.0f * s;
}

// s_waitcnt vmcnt(n) expcnt(7) lgkmcnt(0) (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

// s_waitcnt lgkmcnt(0) only (vector memory loads stay in flight)
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14)); }

#ifndef QG_PINGPONG
#define QG_PINGPONG 1
#endif

// Groups the ping-pong DMA-role step splits its activation DMA into, each followed by a share of
// its dequantisation (0: all loads first, then all dequantisation). Four: step -0.4% against two
// (T=8192 gate/up and down -0.5% / -0.7%, same-box A/B); none: dense +2.5%
#ifndef QG_VMEM_SPLIT
#define QG_VMEM_SPLIT 4
#endif

// ---------------------------------------------------------------------------
// tile kernel
// ---------------------------------------------------------------------------

struct ExpertPtrs {
  const uint8_t* wq[kMaxExpertsPerLaunch];
  const uint16_t* sc[kMaxExpertsPerLaunch];
};

struct TileArgs {
  const uint16_t* x;     // bf16 [rows][K]
  float* y;              // fp32 [out rows][N]
  int M;                 // dense: rows of x and y; MoE: number of assignments (T*topk)
  int N;
  int K;
  // MoE only
  const int32_t* perm;     // assignments grouped by expert
  const int32_t* offsets;  // [E+1] exclusive prefix of per-expert counts
  int e_begin;             // first expert handled by this launch
  int n_experts;           // experts handled by this launch (<= kMaxExpertsPerLaunch)
  int topk;
  int T;
  // dense split-K: `splits` workgroups share a tile, each over a contiguous range of K steps,
  // writing fp32 partials to ws[split][M][N] (summed afterwards in split order)
  float* ws;
  int splits;
  // fused SwiGLU epilogue (MoE gate/up): N = 2 * swi_inter weight rows, h is bf16 [rows][swi_inter]
  int swi_inter;
  uint16_t* h;
  // router-weighted combine fused into the down projection (MoE, y holds the per-slot rows):
  // out[t][n] = sum_j route_w[t*cmb_topk+j] * y[t*cmb_topk+j][n]; arrivals counted per
  // (token, column tile) in counters[T][ceil(N / BN)] (zero at launch)
  int cmb_topk;
  const float* route_w;
  float* out;
  int* counters;
};

// Cache policy of the fused combine's per-slot rows: device scope (sc1), so the stores write
// through this XCD's L2 to the device-coherent level and the loads of the tile that finishes a
// token read what tiles on other XCDs wrote.
constexpr int kDeviceScope = 16;
constexpr int kCmbMaxTopk = 8;   // slots whose loads one thread keeps in flight at once

// Map a linear workgroup id to a tile id so that each XCD (workgroups are
// dispatched round-robin over the 8 XCDs) works on a contiguous tile range
// and neighbouring tiles share operands through that XCD's L2.
__device__ __forceinline__ int xcd_tile(int bid, int ntiles) {
  const int xcd = bid & 7;
  const int local = bid >> 3;
  const int base = ntiles >> 3;
  const int rem = ntiles & 7;
  return xcd * base + (xcd < rem ? xcd : rem) + local;
}

template <int FMT, int BM, int BN, int WM, int WN, bool MOE, int XS = 2>
struct TileKernel {
  static constexpr int kThreads = WM * WN * 64;
  static constexpr int kWaves = WM * WN;
  static constexpr int kWTM = BM / WM;        // rows per wave
  static constexpr int kWTN = BN / WN;        // cols per wave
  static constexpr int kTM = kWTM / 32;       // 32x32 MFMA blocks per wave (M)
  static constexpr int kTN = kWTN / 32;       // (N)
  static constexpr int kXGroups = BM / 8;                         // 8-row groups (1 KiB LDS-DMA loads) per K step
  static constexpr int kXWaves = kXGroups < kWaves ? kXGroups : kWaves;   // waves that issue them
  static constexpr int kXLoads = kXGroups / kXWaves;              // per DMA wave per K step
  static constexpr int kWChunkElems = (FMT == kQ8) ? 16 : 32;   // weights per 16-byte load
  static constexpr int kWChunksPerRow = kBK / kWChunkElems;     // 4 (Q8) or 2 (Q4)
  static constexpr int kWStepBytes = (FMT == kQ8) ? kBK : kBK / 2;   // packed bytes of one row per K step
  static constexpr int kWChunks = BN * kWChunksPerRow / kThreads;
  static constexpr int kXTileBytes = BM * kRowBytes;
  static constexpr int kWTileBytes = BN * kRowBytes;
  static constexpr int kXStages = XS;                            // activation stages (DMA runs XS-1 steps ahead)
  static constexpr int kWBase = XS * kXTileBytes;                 // weight stages follow the activation stages
  static constexpr int kLdsBytes = XS * kXTileBytes + 2 * kWTileBytes;
  static_assert(XS == 2 || XS == 3, "two or three activation stages");
  static_assert(kXLoads * kXWaves * 8 == BM, "x tile must split into 8-row groups per wave");
  static_assert(kWChunks * kThreads == BN * kWChunksPerRow, "w tile must split evenly");
  static_assert(kTM >= 1 && kTN >= 1, "wave tile must hold a 32x32 block");
};

typedef __attribute__((address_space(3))) char lds_char;

// LDS stages of a tile, each its own __shared__ array: the activation DMA of one stage and the
// LDS reads / dequantised-weight writes of the others then have distinct underlying objects, so
// the compiler can tell they do not alias and keeps the DMA in flight across them instead of
// draining it (vmcnt) before every LDS access.
struct LdsStages {
  char* x[3];   // activation stages (x[2] unused with two stages)
  char* w[2];
};

constexpr uint32_t kBufferFlags = 0x00020000;   // raw buffer, 32-bit dwords (gfx9 family)
constexpr uint32_t kOOB = 0xFFFFFFF0u;          // offset past every buffer: loads return 0

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kBufferFlags);
}

#define QG_SG(mask, n) __builtin_amdgcn_sched_group_barrier((mask), (n), 0)
constexpr int kSchedMFMA = 0x008;
constexpr int kSchedVALU = 0x002;
constexpr int kSchedDSRead = 0x100;
constexpr int kSchedDSWrite = 0x200;
#ifndef QG_K_AFTER
#define QG_K_AFTER 1
#endif

// Router-weighted combine fused into the down projection, after a tile has stored its per-slot
// rows (columns [n0, n0 + BN)): each row counts its arrival on (token, column tile); the tile
// whose arrival completes a token's topk slots sums that token's slot rows for these columns in
// increasing slot order (fp32 fused multiply-add from zero, as the standalone combine does, so
// the result is bitwise the same whichever tile finishes it) and writes out[t][n0 .. n0 + BN).
// Every counter reaches topk once per launch sequence; nothing waits for another workgroup.
template <int kThreads, int BM, int BN>
__device__ __forceinline__ void combine_arrivals(const TileArgs& a, __amdgpu_buffer_rsrc_t yr,
                                                 const int* __restrict__ s_yrow, int rows_valid, int n0,
                                                 LdsStages st) {
  typedef __attribute__((address_space(3))) int lds_int;
  const int tid = threadIdx.x;
  const int topk = a.cmb_topk;
  const int N = a.N;
  const int nt_n = (N + BN - 1) / BN;
  const int nt = n0 / BN;
  lds_int* fin = (lds_int*)st.x[0];            // tokens this tile finishes (the K loop is over)
  lds_int* nfin = (lds_int*)st.x[1];
  // this thread's row stores have reached the device-coherent level (and its LDS scratch reads
  // are done); after the barrier every thread's have
  wait_vmcnt_lgkm0<0>();
  __syncthreads();
  if (tid == 0) nfin[0] = 0;
  __syncthreads();
  static_assert(BM <= kThreads, "one thread per tile row");
  if (tid < rows_valid) {
    const int slot = s_yrow[tid];
    if (slot >= 0) {
      const int t = slot / topk;
      const int old = __hip_atomic_fetch_add(a.counters + (size_t)t * nt_n + nt, 1, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
      if (old == topk - 1) fin[__hip_atomic_fetch_add(nfin, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)] = t;
    }
  }
  __syncthreads();
  const int nf = nfin[0];
  const int nc4 = min(BN, N - n0) >> 2;          // 16-byte column chunks of this tile (N % 4 == 0)
  const int items = nf * nc4;
  constexpr int U = 2;                            // (token, chunk) items per thread in flight
  for (int base = 0; base < items; base += U * kThreads) {
    f32x4 acc[U];
    int t_of[U], c_of[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int it = base + u * kThreads + tid;
      t_of[u] = it < items ? fin[it / nc4] : -1;
      c_of[u] = it < items ? n0 + 4 * (it % nc4) : 0;
      acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    for (int j0 = 0; j0 < topk; j0 += kCmbMaxTopk) {
      f32x4 v[U][kCmbMaxTopk];
      float w[U][kCmbMaxTopk];
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < kCmbMaxTopk; ++j) {
          const bool live = t_of[u] >= 0 && j0 + j < topk;
          const int s = live ? t_of[u] * topk + j0 + j : 0;
          w[u][j] = live ? a.route_w[s] : 0.0f;
          v[u][j] = __builtin_bit_cast(
              f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                         yr, live ? ((uint32_t)s * (uint32_t)N + (uint32_t)c_of[u]) * 4u : kOOB, 0, kDeviceScope));
        }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < kCmbMaxTopk; ++j)
          if (j0 + j < topk)
#pragma unroll
            for (int c = 0; c < 4; ++c) acc[u][c] = __builtin_fmaf(w[u][j], v[u][j][c], acc[u][c]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (t_of[u] >= 0)
        __builtin_nontemporal_store(acc[u], reinterpret_cast<f32x4*>(a.out + (size_t)t_of[u] * N + c_of[u]));
  }
}

// One output tile: rows [m0, m0 + rows_valid) of x (dense) or the gathered rows
// s_xrow[] (MoE), columns [n0, n0 + BN) of W.
//
// Pipeline per 64-wide K step kt of the single-barrier tiles (two LDS stages, kWD weight register
// sets; the eight-wave ping-pong loop is described where it is built):
//   issue activation DMA for step kt+1 into stage (kt+1)&1     (buffer_load ... lds)
//   issue packed-weight + scale loads for step kt+kWD          (registers)
//   four K16 sub-steps over stage kt&1: MFMAs, with the next sub-step's LDS
//   fragments and one quarter of step kt+1's dequantisation (into stage
//   (kt+1)&1) interleaved between them
//   wait for the activation DMA and the LDS writes, then barrier
// FULL: every row of the tile is valid, so no MFMA is skipped (branch-free body).
template <int FMT, int BM, int BN, int WM, int WN, bool MOE, bool FULL, int XS, bool SWI, bool CMB>
__device__ __forceinline__ void tile_body(const TileArgs& a, const uint8_t* __restrict__ wq,
                                          const uint16_t* __restrict__ sc, int m0, int n0,
                                          int rows_valid, const int* __restrict__ s_xrow,
                                          const int* __restrict__ s_yrow, LdsStages st,
                                          int ks0, int nsteps, float* __restrict__ yout) {
  using KT = TileKernel<FMT, BM, BN, WM, WN, MOE, XS>;
  static_assert(!SWI || MOE, "the fused SwiGLU epilogue is a MoE gate/up epilogue");
  static_assert(!CMB || (MOE && !SWI), "the fused combine is a MoE down-projection epilogue");
  constexpr int kUnitsPerChunk = (FMT == kQ8) ? 2 : 4;        // 16-byte LDS writes per 16-byte load
  constexpr int kUnits = KT::kWChunks * kUnitsPerChunk;        // per thread per K step
  // weight prefetch distance (K steps): two, and three for the four-wave Q4 tiles (eight-wave Q4
  // tiles at two instead of three: step -1.1%, T=2048 gate/up -2.7%, down -3.5%, T=8192 down -2%,
  // no VGPR spills instead of 9-11 in the 256-row tiles; the four-wave short-prompt tiles
  // 0-1% slower at two; Q8 at three: 108 spills in the dense 256x256 tile)
  constexpr int kWD = (FMT == kQ4 && KT::kWaves == 4) ? 3 : 2;
  // the K loop is unrolled over a period in which activation stage, weight register set and
  // weight LDS stage (two) all repeat
  constexpr int kPeriod = (XS == 3 || kWD == 3) ? 6 : (kWD == 4 ? 4 : 2);
  static_assert(kUnits % 4 == 0, "units must spread evenly over the four K16 sub-steps");
  constexpr int kMfmaPerKK = KT::kTM * KT::kTN;
  constexpr int kValuPerUnit = (FMT == kQ8) ? 20 : 17;

  // Ping-pong (8-wave tiles): the two waves sharing a SIMD belong to different wave rows (wm).
  // Per K step, wm = 1 waves issue the activation DMA while wm = 0 waves run their MFMAs; after
  // a barrier, wm = 1 waves run their MFMAs while wm = 0 waves load and dequantise the next
  // step's weights; a second barrier closes the step. One wave per SIMD issues MFMAs at a time,
  // with its partner's memory and VALU work in the other issue slots, instead of both waves
  // arriving at one barrier at different times.
  constexpr bool PP = QG_PINGPONG && WM == 2 && WN == 4 && XS == 2;
  constexpr int kVmemSplit = QG_VMEM_SPLIT;
  constexpr int XL = PP ? 2 * KT::kXLoads : KT::kXLoads;        // DMA loads per DMA-role wave
  // Weight chunks per thread: without ping-pong every thread takes kWChunks. With it the wm = 0
  // waves take CQ chunks (dequantised after their MFMA phase) and the wm = 1 waves CD chunks
  // (dequantised in their DMA phase).
  // Q4: the wm = 0 waves dequantise every chunk (their phase after the MFMAs had the slack; the
  // DMA role's phase is then the activation DMA and its fragment loads only): 488.7 vs 493.5 us
  // (T=8192 gate/up), 158.1 vs 164.2 us (T=2048 gate/up), same-box A/B; Q8 keeps its 3:1 split
  // (dense 0.8% slower with every chunk on one role)
  constexpr int CQ = PP ? ((FMT == kQ4) ? 2 * KT::kWChunks
                                                       : (KT::kWChunks >= 2 ? (3 * KT::kWChunks + 1) / 2 : KT::kWChunks))
                        : KT::kWChunks;
  constexpr int CD = PP ? 2 * KT::kWChunks - CQ : KT::kWChunks;
  constexpr int WC = CQ > CD ? CQ : CD;                           // register arrays sized for either role
  static_assert(!PP || CQ + CD == 2 * KT::kWChunks, "every chunk dequantised once");
  constexpr int kWStride = PP ? KT::kThreads / 2 : KT::kThreads;
  auto xstage_ptr = [&](int stage) { return (lds_char*)(stage == 0 ? st.x[0] : stage == 1 ? st.x[1] : st.x[2]); };
  auto wstage_ptr = [&](int stage) { return (lds_char*)(stage == 0 ? st.w[0] : st.w[1]); };
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN;
  const int wn = wave % WN;
  const int K = a.K;
  const int N = a.N;
  const int nk = nsteps;          // K steps of this workgroup: absolute steps ks0 .. ks0 + nk - 1
  const uint32_t kblocks = (uint32_t)K >> 5;
  const uint32_t wrow_bytes = (FMT == kQ8) ? (uint32_t)K : (uint32_t)K >> 1;
  const int n_valid = min(BN, N - n0);
  const bool isD = PP ? wm == 1 : true;            // issues activation DMA
  const bool isQ = PP ? wm == 0 : true;            // loads and dequantises weights
  const int xw = PP ? (isD ? wave - WN : 0) : wave;  // DMA wave index within its role
  // 8-row group of the tile fetched by DMA load j of this wave
  auto xgroup = [&](int j) { return xw * XL + j; };
  // first weight chunk of this thread: dequant threads t take chunks t + i * stride (i < CQ), DMA
  // threads t' take CQ * stride + t' + i * stride (i < CD)
  const int wt = PP ? (isQ ? tid : CQ * (KT::kThreads / 2) + (tid - KT::kThreads / 2)) : tid;

  // --- activation DMA: this lane fetches logical chunk dma_c[j] of row (8 g + lane / 8) ---
  __amdgpu_buffer_rsrc_t xr;
  uint32_t xoff[XL];
  int dma_c[XL];
#pragma unroll
  for (int j = 0; j < XL; ++j) {
    const int r = xgroup(j) * 8 + (lane >> 3);
    dma_c[j] = (lane & 7) ^ row_swizzle(r);     // the chunk that lds_chunk(r, .) places at slot lane & 7
  }
  if constexpr (MOE) {
    xr = make_rsrc(a.x, (uint32_t)a.T * (uint32_t)K * 2u);
#pragma unroll
    for (int j = 0; j < XL; ++j) {
      const int r = xgroup(j) * 8 + (lane >> 3);
      const int src = (r < rows_valid) ? s_xrow[r] : -1;
      // a missing row gets an offset that stays past the buffer for every K step's byte offset
      // added to it (the host keeps (T + 1) * K * 2 + 256 below kOOB)
      xoff[j] = (src >= 0) ? (uint32_t)src * (uint32_t)K * 2u + (uint32_t)dma_c[j] * 16u
                           : kOOB - 2u * (uint32_t)K - 2u * (uint32_t)kRowBytes;
    }
  } else {
    xr = make_rsrc(a.x + (size_t)m0 * K, (uint32_t)rows_valid * (uint32_t)K * 2u);
#pragma unroll
    for (int j = 0; j < XL; ++j) {
      const int r = xgroup(j) * 8 + (lane >> 3);
      xoff[j] = (uint32_t)r * (uint32_t)K * 2u + (uint32_t)dma_c[j] * 16u;
    }
  }
  // --- weight / scale offsets of this thread's chunks ---
  // Weight rows of the tile: rows n0 .. n0 + BN - 1, or for the fused SwiGLU epilogue gate/up
  // pairs, tile row 2j -> gate row h0 + j and 2j + 1 -> up row inter + h0 + j (h0 = n0 / 2), so
  // each gate/up pair sits in two neighbouring MFMA columns (lanes). Rows past the matrix read
  // row 0 with a zero scale (SwiGLU) or fall outside the buffer range (plain).
  const int swi_inter = a.swi_inter;
  const int h0 = n0 >> 1;
  const __amdgpu_buffer_rsrc_t wr =
      SWI ? make_rsrc(wq, (uint32_t)N * wrow_bytes) : make_rsrc(wq + (size_t)n0 * wrow_bytes, (uint32_t)n_valid * wrow_bytes);
  const __amdgpu_buffer_rsrc_t sr = SWI ? make_rsrc(sc, (uint32_t)N * kblocks * 2u)
                                        : make_rsrc(sc + (size_t)n0 * kblocks, (uint32_t)n_valid * kblocks * 2u);
  uint32_t woff[WC];
  uint32_t soff[WC];
  int lds_w[WC][kUnitsPerChunk];   // LDS byte offset (within the W tile) of each unit
  int wcol[WC];
  bool wrow_ok[WC];
#pragma unroll
  for (int i = 0; i < WC; ++i) {
    const int q = wt + i * kWStride;
    const int r = q / KT::kWChunksPerRow;
    const int c = q % KT::kWChunksPerRow;
    int grow = r;
    wrow_ok[i] = true;
    if constexpr (SWI) {
      const int hc = h0 + (r >> 1);
      wrow_ok[i] = hc < swi_inter;
      grow = wrow_ok[i] ? ((r & 1) ? swi_inter + hc : hc) : 0;
    }
    wcol[i] = c;
    woff[i] = (uint32_t)grow * wrow_bytes + (uint32_t)c * 16u;
    soff[i] = ((uint32_t)grow * kblocks + (uint32_t)(c * KT::kWChunkElems / 32)) * 2u;
#pragma unroll
    for (int u = 0; u < kUnitsPerChunk; ++u) lds_w[i][u] = lds_chunk(r, c * kUnitsPerChunk + u);
  }

  // Loads of steps past this tile's last one (kt_local >= nk) are issued with out-of-range
  // offsets: the buffer range check answers them with zeros, no memory is read, and the K loop
  // stays free of branches around its loads.
  // A step wholly inside K (every step but a ragged last one and the steps past the end) needs
  // one address add per load; chunks past K and steps past the last one read nothing.
  auto issue_x = [&](int kt_local, int stage, int j0 = 0, int j1 = 1 << 30) {
    const int kt = ks0 + kt_local;
    const uint32_t kbyte = (uint32_t)kt * (uint32_t)kRowBytes;
    const bool tail = (kt + 1) * kBK > K || kt_local >= nk;
    auto issue = [&](bool checked) {
#pragma unroll
      for (int j = 0; j < XL; ++j) {
        if (j < j0 || j >= j1) continue;
        // an 8-row group wholly past the valid rows is not fetched at all: its LDS rows keep
        // stale data, which only reaches accumulator rows that are never stored. (With three
        // stages the waits count this step's activation loads, so every group is issued.)
        if (!FULL && XS == 2 && xgroup(j) * 8 >= rows_valid) continue;
        if (KT::kXWaves < KT::kWaves && xgroup(j) >= KT::kXGroups) continue;   // a wave without DMA
        lds_char* dst = xstage_ptr(stage) + xgroup(j) * 1024;
        if (MOE && !checked) {
          // the step's byte offset rides in the scalar offset: no vector address arithmetic
          // (the row offset alone decides the range check, whether or not the hardware adds
          // the scalar offset to it: missing rows stay past the buffer either way)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (__attribute__((address_space(3))) void*)dst, 16, xoff[j],
                                                   (int)kbyte, 0, 0);
        } else {
          uint32_t off = xoff[j] + kbyte;
          if (checked && (kt_local >= nk || kt * kBK + dma_c[j] * 8 >= K)) off = kOOB;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (__attribute__((address_space(3))) void*)dst, 16, off, 0, 0, 0);
        }
      }
    };
    // (MoE tiles branch on the uniform flag; for dense tiles the branch measured slower than
    // keeping the checks inline)
    if constexpr (MOE) {
      if (tail) issue(true); else issue(false);
    } else {
      issue(tail);
    }
  };

  // weight register sets: the loads of step k are issued kWD steps ahead, into set k % kWD
  uint4 wv[kWD][WC];
  uint32_t sv[kWD][WC];

  auto issue_w = [&](int kt_local, uint4 (&w)[WC], uint32_t (&s)[WC], int cnt, int i0 = 0) {
    const int kt = ks0 + kt_local;
    const bool live = kt_local < nk;
#pragma unroll
    for (int i = 0; i < WC; ++i) {
      if (i >= cnt) break;
      if (i < i0) continue;
      const uint32_t wo = live ? woff[i] + (uint32_t)kt * KT::kWStepBytes : kOOB;
      const uint32_t so = live ? soff[i] + (uint32_t)kt * 4u : kOOB;
      w[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(wr, wo, 0, 0));
      s[i] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(sr, so, 0, 0);
    }
  };

  // dequantise unit u (0 <= u < kUnits) of a weight register set into LDS stage `stage`
  // Q8: scl = s; Q4: scl = s * 2^24, scl16 = s * 2^20, soffv = -8 s (dequant_q4_unit)
  float scl[WC], scl16[WC], soffv[WC];
  auto dequant_unit = [&](int kt, int u, const uint4 (&w)[WC], const uint32_t (&s)[WC], int stage) {
    const int i = u / kUnitsPerChunk;
    const int sub = u % kUnitsPerChunk;
    if (sub == 0) {
      const bool valid = wrow_ok[i] && (ks0 + kt) * kBK + wcol[i] * KT::kWChunkElems < K;
      scl[i] = valid ? fp16_to_f32((uint16_t)s[i]) : 0.0f;
      if constexpr (FMT == kQ4) q4_factors(scl[i], scl[i], scl16[i], soffv[i]);
    }
    const uint32_t d[4] = {w[i].x, w[i].y, w[i].z, w[i].w};
    u32x4 o;
    if constexpr (FMT == kQ8)
      o = dequant_q8_unit(d[2 * sub], d[2 * sub + 1], scl[i]);
    else
      o = dequant_q4_unit(d[sub], scl[i], scl16[i], soffv[i]);
    *reinterpret_cast<lds_u32x4*>(wstage_ptr(stage) + lds_w[i][sub]) = o;
  };

  f32x16 acc[KT::kTM][KT::kTN];
#pragma unroll
  for (int i = 0; i < KT::kTM; ++i)
#pragma unroll
    for (int j = 0; j < KT::kTN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // 32-row block i of this wave is tile block i * WM + wm (blocks dealt round-robin over the
  // WM wave rows, so a partly filled tile spreads its valid blocks evenly over the waves)
  const int nvalid_blocks = (rows_valid + 31) >> 5;
  const int mblocks = FULL ? KT::kTM : (nvalid_blocks > wm ? (nvalid_blocks - wm + WM - 1) / WM : 0);
  const int lr = lane & 31;
  const int lh = lane >> 5;
  // per-lane LDS byte offsets of the A / B fragments of sub-step 0 (chunk lh); chunk 2 kk + lh
  // of row r sits at r * 128 + (((2 kk + lh) ^ row_swizzle(r)) << 4)
  int aoff[KT::kTM], boff[KT::kTN];
#pragma unroll
  for (int i = 0; i < KT::kTM; ++i) aoff[i] = ((i * WM + wm) * 32 + lr) * kRowBytes;
#pragma unroll
  for (int j = 0; j < KT::kTN; ++j) boff[j] = (wn * KT::kWTN + j * 32 + lr) * kRowBytes;
  const int rsw = row_swizzle(lr);   // the same for every fragment row: bases are multiples of 32 (16 would do)

  // Fragment registers: sub-step kk uses set kk & 1. The last sub-step's MFMAs run after
  // the barrier that closes the K step, overlapping the next step's first LDS reads.
  bf16x8 av[2][KT::kTM], bv[2][KT::kTN];
  auto load_frags = [&](int xstage, int wstage, int kk, int buf) {
    const lds_char* xs = xstage_ptr(xstage);
    const lds_char* ws = wstage_ptr(wstage);
    const int slot = ((kk * 2 + lh) ^ rsw) << 4;
#pragma unroll
    for (int j = 0; j < KT::kTN; ++j)
      bv[buf][j] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8*>(ws + boff[j] + slot);
#pragma unroll
    for (int i = 0; i < KT::kTM; ++i)
      av[buf][i] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8*>(xs + aoff[i] + slot);
  };
  auto mfmas = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KT::kTM; ++i) {
      if (FULL || i < mblocks) {
#pragma unroll
        for (int j = 0; j < KT::kTN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[buf][i], bv[buf][j], acc[i][j], 0, 0, 0);
      }
    }
  };
  // The MFMAs of the last kAfter sub-steps of a step run after the barrier that closes it, so a
  // wave that reaches the barrier early still has that much matrix work queued behind it.
  constexpr int kAfter = QG_K_AFTER;
  constexpr int kHead = 4 - kAfter;                  // sub-steps whose MFMAs run before the barrier
  // dequantisation units of the next step, spread over the head sub-steps (they must land before
  // the barrier)
  constexpr int kUnitGroups = kHead;
  auto unit_lo = [](int kk) { return (kk * kUnits + kUnitGroups - 1) / kUnitGroups; };

  // head of step kt over activation stage xcur and weight stage wcur (fragments of sub-step 0
  // already in set 0), with step kt+1's weights (set wn_) dequantised into weight stage wcur ^ 1;
  // leaves the fragments of the last kAfter sub-steps in their sets (sub-step kk in set kk & 1)
  auto step_head = [&](int kt, int xcur, int wcur, const uint4 (&wn_)[WC], const uint32_t (&sn_)[WC]) {
#pragma unroll
    for (int kk = 0; kk < kHead; ++kk) {
      const int buf = kk & 1;
      load_frags(xcur, wcur, kk + 1, buf ^ 1);
      mfmas(buf);
      // step kt+1's weights (on the last step this writes the idle stage with unused data:
      // harmless, and it keeps the body branch-free for the MFMA/VALU interleave)
#pragma unroll
      for (int u = unit_lo(kk); u < unit_lo(kk + 1); ++u) dequant_unit(kt + 1, u, wn_, sn_, wcur ^ 1);
      if constexpr (FULL) {
        constexpr int kUnitsHere = kUnits / kUnitGroups + 1;
        constexpr int kVpm = (kUnitsHere * kValuPerUnit + 4 + kMfmaPerKK - 1) / kMfmaPerKK;
        QG_SG(kSchedMFMA, 1);
        QG_SG(kSchedDSRead, KT::kTM + KT::kTN);
#pragma unroll
        for (int m = 1; m < kMfmaPerKK; ++m) {
          QG_SG(kSchedVALU, kVpm);
          QG_SG(kSchedMFMA, 1);
        }
        QG_SG(kSchedVALU, kVpm);
        QG_SG(kSchedDSWrite, kUnitsHere);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // with two sub-steps after the barrier, sub-step 3's fragments load into the set that
    // sub-step 1's MFMAs (just issued) read
    if constexpr (kAfter == 2) {
      load_frags(xcur, wcur, 3, 1);
      if constexpr (FULL) __builtin_amdgcn_sched_barrier(0);
    }
  };
  // after the barrier: the last kAfter sub-steps' MFMAs, with the next step's sub-step 0
  // fragments (if any) loaded into set 0 once the MFMAs reading set 0 have issued
  auto step_tail = [&](bool next, int next_xstage, int next_wstage) {
    if constexpr (kAfter == 2) {
      mfmas(0);
      if constexpr (FULL) __builtin_amdgcn_sched_barrier(0);
      if (next) load_frags(next_xstage, next_wstage, 0, 0);
      mfmas(1);
    } else {
      if (next) load_frags(next_xstage, next_wstage, 0, 0);
      mfmas(1);
    }
    if constexpr (FULL) __builtin_amdgcn_sched_barrier(0);
  };

  if constexpr (!PP) {
    // prologue: steps 0 .. XS-2 of the activations and steps 0 .. kWD-1 of the weights in flight;
    // step 0's weights dequantised into weight stage 0
    constexpr int kAhead = XS - 1;                              // activation prefetch distance (steps)
    // vmcnt retires in issue order, so waiting for a weight register set also waits for every
    // load issued before it: with three activation stages the weights of a step are issued
    // before its activations, so dequantising them never forces the younger activations.
    // The order of the loads in flight is pinned with scheduling barriers: the waits below count
    // the loads issued after a given activation step, which is only exact if the compiler keeps
    // every group of loads where it is written. Weight loads of steps beyond the last one read
    // inside the buffer range or are cut off by it (zeros), so they are issued unconditionally.
    issue_x(0, 0);
    __builtin_amdgcn_sched_barrier(0);
  #pragma unroll
    for (int k = 0; k < kWD; ++k) issue_w(k, wv[k], sv[k], WC);
    __builtin_amdgcn_sched_barrier(0);
    if (XS == 3) issue_x(1, 1);
    __builtin_amdgcn_sched_barrier(0);
  #pragma unroll
    for (int u = 0; u < kUnits; ++u) dequant_unit(0, u, wv[0], sv[0], 0);
    // step 0's activations landed: allow what was issued after them to stay in flight
    // Weight loads whose registers are never read again (steps past the last one, j > nk) may be
    // deleted by the compiler, so a wait counts only the weight loads that are certainly issued
    // (j <= nk): an undercount only makes the wait stricter.
    {
      const int w_live = min(kWD, nk + 1);
      constexpr int kX1 = XS == 3 ? KT::kXLoads : 0;
      if (w_live >= 3) wait_vmcnt_lgkm0<3 * 2 * KT::kWChunks + kX1>();
      else if (w_live == 2) wait_vmcnt_lgkm0<2 * 2 * KT::kWChunks + kX1>();
      else wait_vmcnt_lgkm0<2 * KT::kWChunks + kX1>();
    }
    __builtin_amdgcn_s_barrier();
    load_frags(0, 0, 0, 0);

    // Step kt (S = kt % kPeriod): issue the activations of step kt + kAhead and the weights of
    // step kt + kWD, MFMA over activation stage kt % XS / weight stage kt & 1 while step kt+1's
    // weights (register set (kt+1) % kWD) are dequantised into weight stage (kt+1) & 1, then wait
    // for step kt+1's activations and close the step with a barrier.
    auto step = [&](auto S_, int kt) {
      constexpr int S = decltype(S_)::value;
      constexpr int xs_cur = S % XS, xs_next = (S + 1) % XS, xs_ahead = (S + kAhead) % XS;
      constexpr int wset_issue = S % kWD, wset_next = (S + 1) % kWD;
      if (XS == 2) issue_x(kt + kAhead, xs_ahead);
      __builtin_amdgcn_sched_barrier(0);
      issue_w(kt + kWD, wv[wset_issue], sv[wset_issue], WC);
      __builtin_amdgcn_sched_barrier(0);
      if (XS == 3) issue_x(kt + kAhead, xs_ahead);
      __builtin_amdgcn_sched_barrier(0);
      step_head(kt, xs_cur, S & 1, wv[wset_next], sv[wset_next]);
      // loads issued after x(kt+1): XS == 2 -> this step's weights; XS == 3 -> this step's
      // weights and activations (x(kt+1) was issued one step earlier)
      // (weight loads of steps past the last one may be deleted: counted only when live)
      const bool w_live = kt + kWD <= nk;
      if constexpr (XS == 3) {
        if (w_live) wait_vmcnt_lgkm0<2 * KT::kWChunks + KT::kXLoads>(); else wait_vmcnt_lgkm0<KT::kXLoads>();
      } else {
        if (w_live) wait_vmcnt_lgkm0<2 * KT::kWChunks>(); else wait_vmcnt_lgkm0<0>();
      }
      __builtin_amdgcn_s_barrier();
      step_tail(kt + 1 < nk, xs_next, (S + 1) & 1);
    };
    int kt = 0;
    // whole periods, then the remaining steps (each guarded by the step count)
    auto period = [&]<int... S>(std::integer_sequence<int, S...>) {
      for (; kt + kPeriod <= nk; kt += kPeriod) (step(std::integral_constant<int, S>{}, kt + S), ...);
      ((kt + S < nk && S < kPeriod - 1 ? (step(std::integral_constant<int, S>{}, kt + S), 0) : 0), ...);
    };
    period(std::make_integer_sequence<int, kPeriod>{});
  } else {
    // ---- ping-pong K loop (see PP above) ----
    // One wave's MFMAs for a whole step: fragments of sub-step kk+1 load while sub-step kk's
    // MFMAs run; sub-step 0's fragments are already in set 0 when `pre` is set.
    auto mfma_phase = [&](int xst, int wst, bool pre) {
      if (!pre) load_frags(xst, wst, 0, 0);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        if (kk < 3) load_frags(xst, wst, kk + 1, (kk + 1) & 1);
        mfmas(kk & 1);
        if constexpr (FULL) {
          QG_SG(kSchedMFMA, 1);
          if (kk < 3) QG_SG(kSchedDSRead, KT::kTM + KT::kTN);
          QG_SG(kSchedMFMA, kMfmaPerKK - 1);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    };
    // prologue: activations of step 0 (DMA waves), weights of steps 0 .. kWD-1 in flight and
    // step 0's dequantised into weight stage 0 (dequant waves)
    if (isD) {
      issue_x(0, 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int k = 0; k < kWD; ++k) issue_w(k, wv[k], sv[k], CD);
#pragma unroll
      for (int u = 0; u < CD * kUnitsPerChunk; ++u) dequant_unit(0, u, wv[0], sv[0], 0);
      wait_vmcnt_lgkm0<0>();
    } else {
#pragma unroll
      for (int k = 0; k < kWD; ++k) issue_w(k, wv[k], sv[k], CQ);
#pragma unroll
      for (int u = 0; u < CQ * kUnitsPerChunk; ++u) dequant_unit(0, u, wv[0], sv[0], 0);
      // a dequant wave waits for its LDS writes only (its weight registers are waited on where
      // they are read)
      wait_lgkm0();
    }
    __builtin_amdgcn_s_barrier();

    // The two roles run separate loops (the role branch taken once, outside the K loop, so the
    // accumulators never meet at a join); both execute two barriers per step.
    auto q_step = [&](auto S_, int kt) {
      constexpr int S = decltype(S_)::value;
      constexpr int xs_cur = S % 2, ws_cur = S & 1;
      constexpr int wset_issue = S % kWD, wset_next = (S + 1) % kWD;
      mfma_phase(xs_cur, ws_cur, false);                   // stage kt complete since the last barrier
      __builtin_amdgcn_s_barrier();
      if constexpr (kVmemSplit > 0) {
        // weight loads chunk by chunk, each followed by the dequantisation of one chunk of the
        // other register set (the set of step kt, dequantised last step, receives step kt+kWD)
#pragma unroll
        for (int i = 0; i < CQ; ++i) {
          issue_w(kt + kWD, wv[wset_issue], sv[wset_issue], i + 1, i);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int u = i * kUnitsPerChunk; u < (i + 1) * kUnitsPerChunk; ++u)
            dequant_unit(kt + 1, u, wv[wset_next], sv[wset_next], ws_cur ^ 1);
          __builtin_amdgcn_sched_barrier(0);
        }
      } else {
        issue_w(kt + kWD, wv[wset_issue], sv[wset_issue], CQ);  // the set of step kt, dequantised last step
#pragma unroll
        for (int u = 0; u < CQ * kUnitsPerChunk; ++u)
          dequant_unit(kt + 1, u, wv[wset_next], sv[wset_next], ws_cur ^ 1);
      }
      wait_lgkm0();
      __builtin_amdgcn_s_barrier();
    };
    auto d_step = [&](auto S_, int kt) {
      constexpr int S = decltype(S_)::value;
      constexpr int xs_cur = S % 2, xs_next = (S + 1) % 2, ws_cur = S & 1;
      constexpr int wset_issue = S % kWD, wset_next = (S + 1) % kWD;
      constexpr int NU = CD * kUnitsPerChunk;              // dequantisation units of this wave
      // The activation DMA (stage last read in step kt-1) goes out in kVmemSplit groups with a
      // share of the dequantisation after each, so the wave works while its loads queue in the
      // address unit. The vector-memory order is unchanged: all DMA groups, then the weight
      // loads (the wait at the end of the step counts the loads after the DMA).
      constexpr int G = kVmemSplit > 0 ? kVmemSplit : 1;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        issue_x(kt + 1, xs_next, g * XL / G, (g + 1) * XL / G);
        __builtin_amdgcn_sched_barrier(0);
        if (g == G - 1) {
          issue_w(kt + kWD, wv[wset_issue], sv[wset_issue], CD);
          __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (kVmemSplit > 0) {
#pragma unroll
          for (int u = g * NU / G; u < (g + 1) * NU / G; ++u)
            dequant_unit(kt + 1, u, wv[wset_next], sv[wset_next], ws_cur ^ 1);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      if constexpr (kVmemSplit == 0) {
#pragma unroll
        for (int u = 0; u < NU; ++u)
          dequant_unit(kt + 1, u, wv[wset_next], sv[wset_next], ws_cur ^ 1);
      }
      load_frags(xs_cur, ws_cur, 0, 0);                    // prefetch for the MFMA phase
      __builtin_amdgcn_s_barrier();
      mfma_phase(xs_cur, ws_cur, true);
      // this wave's activation DMA of step kt+1: the only vector-memory loads issued after it are
      // its weight loads of step kt+kWD, counted only when live (loads of steps past the last one
      // may be deleted, and an undercount only makes the wait stricter)
      if (kt + kWD <= nk) wait_vmcnt_lgkm0<2 * CD>(); else wait_vmcnt_lgkm0<0>();
      __builtin_amdgcn_s_barrier();
    };
    int kt = 0;
    if (isQ) {
      auto period = [&]<int... S>(std::integer_sequence<int, S...>) {
        for (; kt + kPeriod <= nk; kt += kPeriod) (q_step(std::integral_constant<int, S>{}, kt + S), ...);
        ((kt + S < nk && S < kPeriod - 1 ? (q_step(std::integral_constant<int, S>{}, kt + S), 0) : 0), ...);
      };
      period(std::make_integer_sequence<int, kPeriod>{});
    } else {
      auto period = [&]<int... S>(std::integer_sequence<int, S...>) {
        for (; kt + kPeriod <= nk; kt += kPeriod) (d_step(std::integral_constant<int, S>{}, kt + S), ...);
        ((kt + S < nk && S < kPeriod - 1 ? (d_step(std::integral_constant<int, S>{}, kt + S), 0) : 0), ...);
      };
      period(std::make_integer_sequence<int, kPeriod>{});
    }
  }
  // only out-of-range loads (past the last step) can still be in flight: retire them before the
  // workgroup can end
  wait_vmcnt_lgkm0<0>();

  // --- epilogue: lane holds column (lane & 31) and rows (r/4)*8 + (lane/32)*4 + r%4 of each block ---
  if constexpr (SWI) {
    // Lanes 2k (gate) and 2k + 1 (up) hold the pair of h column h0 + (tile column) / 2 for the
    // same 16 rows. One exchange per row pair splits the work: the even lane keeps rows q
    // (0 <= q < 8) and receives their up values, the odd lane keeps rows q + 8 and receives their
    // gate values, so every lane evaluates the SiLU gate for 8 rows and stores them.
    const bool odd = (lr & 1) != 0;
    // Staged path: a wave's h columns (h0 + wn * kWTN / 2 + [0, kWTN / 2)) all valid and rows
    // 16-byte aligned: h values go through a per-wave LDS scratch and leave as 16-byte row chunks
    // (8 bf16); the K loop ends with a barrier after its last LDS access.
    constexpr int kHW = KT::kWTN / 2;             // h columns per wave
    static_assert(kHW % 8 == 0, "whole 16-byte chunks per wave row");
    if ((swi_inter & 7) == 0 && h0 + (wn + 1) * kHW <= swi_inter) {
      constexpr int kStrideH = kHW + 8;           // bf16 per scratch row (16-byte aligned rows)
      constexpr int kHalf = KT::kWaves / 2;
      // half of the waves per LDS stage: the activation stages, or the weight stages when an
      // activation stage is too small (short tiles)
      constexpr int kNeed = kHalf * 32 * kStrideH * 2;
      constexpr bool kInX = kNeed <= KT::kXTileBytes;
      static_assert(kInX || kNeed <= KT::kWTileBytes, "epilogue scratch must fit an LDS stage");
      lds_char* scratch = (kInX ? xstage_ptr(wave / kHalf) : wstage_ptr(wave / kHalf)) + (wave % kHalf) * (32 * kStrideH * 2);
      constexpr int kChunksRow = kHW / 8;
#pragma unroll
      for (int i = 0; i < KT::kTM; ++i) {
        if (!FULL && i >= mblocks) continue;
#pragma unroll
        for (int j = 0; j < KT::kTN; ++j) {
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float lo = acc[i][j][q];
            const float hi = acc[i][j][q + 8];
            const float recv = __builtin_bit_cast(
                float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, odd ? lo : hi), 0xB1, 0xF, 0xF, false));
            const float g = odd ? recv : lo;
            const float u = odd ? hi : recv;
            const int rm = odd ? q + 8 : q;
            const int row = (rm >> 2) * 8 + lh * 4 + (rm & 3);
            const int hcol = j * 16 + (lr >> 1);
            *reinterpret_cast<__attribute__((address_space(3))) uint16_t*>(scratch + (row * kStrideH + hcol) * 2) =
                (uint16_t)(pack_bf16x2(swiglu_f32(g, u), 0.0f) & 0xFFFFu);
          }
        }
        const int rbase = (i * WM + wm) * 32;
#pragma unroll
        for (int g = 0; g < 32 * kChunksRow / 64; ++g) {
          const int idx = g * 64 + lane;
          const int row = idx / kChunksRow;
          const int ch = idx % kChunksRow;
          const u32x4 v = *reinterpret_cast<const lds_u32x4*>(scratch + (row * kStrideH + ch * 8) * 2);
          const int trow = rbase + row;
          if (!FULL && trow >= rows_valid) continue;
          const int dst = s_yrow[trow];
          if (dst < 0) continue;
          *reinterpret_cast<u32x4*>(a.h + (size_t)dst * swi_inter + h0 + wn * kHW + ch * 8) = v;
        }
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < KT::kTM; ++i) {
      if (!FULL && i >= mblocks) continue;
#pragma unroll
      for (int j = 0; j < KT::kTN; ++j) {
        const int hc = h0 + ((wn * KT::kWTN + j * 32 + lr) >> 1);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const float lo = acc[i][j][q];
          const float hi = acc[i][j][q + 8];
          // DPP quad_perm [1,0,3,2]: the value of lane l ^ 1 (both lanes active)
          const float recv = __builtin_bit_cast(
              float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, odd ? lo : hi), 0xB1, 0xF, 0xF, false));
          const float g = odd ? recv : lo;
          const float u = odd ? hi : recv;
          const int rm = odd ? q + 8 : q;
          const int row = (i * WM + wm) * 32 + (rm >> 2) * 8 + lh * 4 + (rm & 3);
          if (!FULL && row >= rows_valid) continue;
          const int dst = s_yrow[row];
          if (dst >= 0 && hc < swi_inter)
            a.h[(size_t)dst * swi_inter + hc] = (uint16_t)(pack_bf16x2(swiglu_f32(g, u), 0.0f) & 0xFFFFu);
        }
      }
    }
    return;
  }
  const bool full_cols = n0 + BN <= N;
  // fused combine: per-slot rows leave with device-scope stores (32-bit offsets: the host checks
  // that y spans less than 4 GiB)
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(yout, CMB ? (uint32_t)((size_t)a.M * (size_t)N * 4u) : 0u);
  auto store_row4 = [&](int dst, int col, const f32x4& v) {
    if constexpr (CMB)
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), yr, ((uint32_t)dst * (uint32_t)N + (uint32_t)col) * 4u,
                                             0, kDeviceScope);
    else
      *reinterpret_cast<f32x4*>(yout + (size_t)dst * N + col) = v;
  };
  auto store_one = [&](int dst, int col, float v) {
    if constexpr (CMB)
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), yr,
                                            ((uint32_t)dst * (uint32_t)N + (uint32_t)col) * 4u, 0, kDeviceScope);
    else
      yout[(size_t)dst * N + col] = v;
  };
  if (full_cols && (N & 3) == 0) {
    // Row-contiguous stores through LDS: each 32x32 accumulator block goes to a per-wave LDS
    // scratch (row stride 40 floats: the two row halves a store instruction writes fall in
    // disjoint banks) and comes back as 16-byte row chunks, so a wave stores a block with 4
    // dwordx4 instructions instead of 16 dword ones. Every wave is past its last LDS read of the
    // K loop (the loop ends with a barrier after the last fragment reads and DMA waits).
    constexpr int kStride = 40;
    constexpr int kHalf = KT::kWaves / 2;
    constexpr int kNeed = kHalf * 32 * kStride * 4;
    constexpr bool kInX = kNeed <= KT::kXTileBytes;
    static_assert(kInX || kNeed <= KT::kWTileBytes, "epilogue scratch must fit an LDS stage");
    lds_char* scratch = (kInX ? xstage_ptr(wave / kHalf) : wstage_ptr(wave / kHalf)) + (wave % kHalf) * (32 * kStride * 4);
    const int rr = lane >> 3;                 // row within an 8-row read group
    const int cc = (lane & 7) * 4;            // first of this lane's 4 columns
#pragma unroll
    for (int i = 0; i < KT::kTM; ++i) {
      if (!FULL && i >= mblocks) continue;
      const int rbase = (i * WM + wm) * 32;
#pragma unroll
      for (int j = 0; j < KT::kTN; ++j) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = (r >> 2) * 8 + lh * 4 + (r & 3);
          *reinterpret_cast<__attribute__((address_space(3))) float*>(scratch + (row * kStride + lr) * 4) =
              acc[i][j][r];
        }
        const int col = n0 + wn * KT::kWTN + j * 32 + cc;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int row = g * 8 + rr;
          const f32x4 v =
              *reinterpret_cast<const __attribute__((address_space(3))) f32x4*>(scratch + (row * kStride + cc) * 4);
          const int trow = rbase + row;
          if (!FULL && trow >= rows_valid) continue;
          const int dst = MOE ? s_yrow[trow] : (m0 + trow);
          if (MOE && dst < 0) continue;
          store_row4(dst, col, v);
        }
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < KT::kTM; ++i) {
      if (!FULL && i >= mblocks) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = (i * WM + wm) * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
        if (!FULL && row >= rows_valid) continue;
        const int dst = MOE ? s_yrow[row] : (m0 + row);
        if (MOE && dst < 0) continue;
        const int col0 = n0 + wn * KT::kWTN + lr;
#pragma unroll
        for (int j = 0; j < KT::kTN; ++j)
          if (full_cols || col0 + j * 32 < N) store_one(dst, col0 + j * 32, acc[i][j][r]);
      }
    }
  }
  if constexpr (CMB) combine_arrivals<KT::kThreads, BM, BN>(a, yr, s_yrow, rows_valid, n0, st);
}

template <int FMT, int BM, int BN, int WM, int WN, bool MOE, int XS, bool SWI, bool CMB = false>
__device__ __forceinline__ void tile_dispatch(const TileArgs& a, const uint8_t* __restrict__ wq,
                                              const uint16_t* __restrict__ sc, int m0, int n0, int rows_valid,
                                              const int* __restrict__ s_xrow, const int* __restrict__ s_yrow,
                                              LdsStages lds, int ks0, int nsteps, float* __restrict__ yout) {
  if (rows_valid == BM)
    tile_body<FMT, BM, BN, WM, WN, MOE, true, XS, SWI, CMB>(a, wq, sc, m0, n0, rows_valid, s_xrow, s_yrow, lds, ks0,
                                                            nsteps, yout);
  else
    tile_body<FMT, BM, BN, WM, WN, MOE, false, XS, SWI, CMB>(a, wq, sc, m0, n0, rows_valid, s_xrow, s_yrow, lds, ks0,
                                                             nsteps, yout);
}

template <int FMT, int BM, int BN, int WM, int WN, int XS>
__global__ __launch_bounds__(WM * WN * 64) void dense_kernel(TileArgs a, const uint8_t* __restrict__ wq,
                                                             const uint16_t* __restrict__ sc) {
  using KT = TileKernel<FMT, BM, BN, WM, WN, false, XS>;
  __shared__ __attribute__((aligned(1024))) char lx0[KT::kXTileBytes];
  __shared__ __attribute__((aligned(1024))) char lx1[KT::kXTileBytes];
  __shared__ __attribute__((aligned(1024))) char lx2[XS == 3 ? KT::kXTileBytes : 16];
  __shared__ __attribute__((aligned(1024))) char lw0[KT::kWTileBytes];
  __shared__ __attribute__((aligned(1024))) char lw1[KT::kWTileBytes];
  const LdsStages lds{{lx0, lx1, XS == 3 ? lx2 : nullptr}, {lw0, lw1}};
  const int mt_n = (a.M + BM - 1) / BM;
  const int nt_n = (a.N + BN - 1) / BN;
  const int ntiles = mt_n * nt_n;
  const int split = (int)blockIdx.x / ntiles;
  const int tile = xcd_tile((int)blockIdx.x - split * ntiles, ntiles);
  // column-tile major: consecutive tiles (same XCD) share a weight column tile
  const int nt = tile / mt_n;
  const int mt = tile - nt * mt_n;
  const int m0 = mt * BM;
  const int rows_valid = min(BM, a.M - m0);
  const int nk_all = (a.K + kBK - 1) / kBK;
  const int per = (nk_all + a.splits - 1) / a.splits;
  const int ks0 = split * per;
  const int nsteps = min(per, nk_all - ks0);
  float* yout = a.splits > 1 ? a.ws + (size_t)split * a.M * a.N : a.y;
  tile_dispatch<FMT, BM, BN, WM, WN, false, XS, false>(a, wq, sc, m0, nt * BN, rows_valid, nullptr, nullptr, lds, ks0,
                                                       nsteps, yout);
}

// Grouped MoE GEMM: the launch covers experts [e_begin, e_begin + n_experts).
// Work items are (expert, m tile, n tile) over active experts only; every
// workgroup decodes its item from the per-expert counts, so the host never
// needs the routing.
template <int FMT, int BM, int BN, int WM, int WN, int XS, bool SWI, bool CMB = false>
// four-wave 128x128 tiles (67 KB of LDS) run two workgroups per CU (at most 256 registers per
// lane), four-wave 64x128 tiles (50 KB) three
__global__ __launch_bounds__(WM * WN * 64, WM * WN == 4 ? (BM <= 64 ? 3 : 2) : 1) void moe_kernel(TileArgs a,
                                                                                                  ExpertPtrs ep) {
  using KT = TileKernel<FMT, BM, BN, WM, WN, true, XS>;
  static_assert(KT::kThreads >= kMaxExpertsPerLaunch, "the tile prefix needs one lane per expert");
  __shared__ __attribute__((aligned(1024))) char lx0[KT::kXTileBytes];
  __shared__ __attribute__((aligned(1024))) char lx1[KT::kXTileBytes];
  __shared__ __attribute__((aligned(1024))) char lx2[XS == 3 ? KT::kXTileBytes : 16];
  __shared__ __attribute__((aligned(1024))) char lw0[KT::kWTileBytes];
  __shared__ __attribute__((aligned(1024))) char lw1[KT::kWTileBytes];
  const LdsStages lds{{lx0, lx1, XS == 3 ? lx2 : nullptr}, {lw0, lw1}};
  __shared__ int s_prefix[kMaxExpertsPerLaunch + 1];
  __shared__ int s_rowidx[BM];   // y row (assignment) of each tile row
  __shared__ int s_xrow[BM];     // x row (token = assignment / topk) of each tile row
  const int tid = threadIdx.x;
  // fused SwiGLU: a tile covers BN / 2 columns of h (BN interleaved gate/up weight rows)
  const int nt_n = SWI ? (a.swi_inter + BN / 2 - 1) / (BN / 2) : (a.N + BN - 1) / BN;
  const int ne = a.n_experts;

  // per-expert m-tile counts -> inclusive prefix over the launch's experts (<= 128):
  // one expert per lane of the first two waves, wave prefix sums, then combine.
  __shared__ int s_wsum[2];
  if (tid < 128) {
    int mtiles = 0;
    if (tid < ne) {
      const int lo = a.offsets[a.e_begin + tid];
      const int hi = a.offsets[a.e_begin + tid + 1];
      int c = hi - lo;
      if (lo < 0 || hi > a.M || c < 0) c = 0;   // inconsistent table: no work for this expert
      mtiles = (c + BM - 1) / BM;
    }
    int incl = mtiles;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int v = __shfl_up(incl, d, 64);
      if ((tid & 63) >= d) incl += v;
    }
    if ((tid & 63) == 63) s_wsum[tid >> 6] = incl;
    s_prefix[tid + 1] = incl;
    if (tid == 0) s_prefix[0] = 0;
  }
  __syncthreads();
  if (tid >= 64 && tid < 128) s_prefix[tid + 1] += s_wsum[0];
  __syncthreads();
  // Work unit: an m-tile group = one expert's BM gathered rows against all nt_n column tiles.
  // Workgroups reach the 8 XCDs round-robin (bid % 8). Groups are dealt to the XCDs in runs of
  // kMoeRun consecutive groups (XCD x takes runs x, x + 8, ...), so heavy and light groups (skewed
  // routing) spread evenly over the XCDs while the groups of one run -- mostly the same expert --
  // share an L2. Inside a run the workgroups go column tile by column tile, the run's groups
  // innermost: neighbouring workgroups read the same weight column tile, and each group's gathered
  // rows serve its nt_n column tiles within a window of kMoeRun * nt_n workgroups.
  // The host sizes the grid as 8 * kMoeRun * ceil(groups bound / (8 * kMoeRun)) * nt_n.
  const int ngroups = s_prefix[ne];
  const int xcd = (int)blockIdx.x & 7;
  const int local = (int)blockIdx.x >> 3;
  const int run = local / (kMoeRun * nt_n);
  const int within = local - run * (kMoeRun * nt_n);
  const int nt = within / kMoeRun;
  const int g = (run * 8 + xcd) * kMoeRun + (within - nt * kMoeRun);
  if (g >= ngroups) return;
  // largest e with s_prefix[e] <= g
  int lo = 0, hi = ne;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (s_prefix[mid] <= g) lo = mid; else hi = mid;
  }
  const int e = lo;
  const int mt = g - s_prefix[e];
  const int pbeg = a.offsets[a.e_begin + e] + mt * BM;
  const int pend = a.offsets[a.e_begin + e + 1];
  const int rows_valid = min(BM, pend - pbeg);
  for (int r = tid; r < BM; r += KT::kThreads) {
    int asg = -1;
    if (r < rows_valid) {
      asg = a.perm[pbeg + r];
      if (asg < 0 || asg >= a.M) asg = -1;
    }
    s_rowidx[r] = asg;
    s_xrow[r] = asg < 0 ? -1 : asg / a.topk;
  }
  __syncthreads();
  const int nk = (a.K + kBK - 1) / kBK;
  if constexpr (WM == 2 && WN == 4) {
    // A group of at most 32 rows (a small expert, or the last rows of a large one) has MFMA work
    // for one wave row only, while the whole tile's weights still need dequantising: such a tile
    // runs as 32 rows by BN over all eight waves side by side, each dequantising an eighth of the
    // weights, on the single-barrier loop (same products in the same order, so the same bits).
    if (rows_valid <= 32) {
      tile_dispatch<FMT, 32, BN, 1, 8, true, 2, SWI, CMB>(a, ep.wq[e], ep.sc[e], 0, nt * BN, rows_valid, s_xrow,
                                                         s_rowidx, lds, 0, nk, a.y);
      return;
    }
  }
  tile_dispatch<FMT, BM, BN, WM, WN, true, XS, SWI, CMB>(a, ep.wq[e], ep.sc[e], 0, nt * BN, rows_valid, s_xrow,
                                                         s_rowidx, lds, 0, nk, a.y);
}

}  // namespace qg
