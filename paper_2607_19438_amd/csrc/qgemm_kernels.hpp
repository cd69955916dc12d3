// Device code of the block-quantised prefill GEMM for gfx950 (MI355X).
//
// One workgroup owns one output tile and walks the contraction dimension,
// accumulating tile products into register-resident fp32 accumulators (the
// structure Section 3.1 describes for the paper's matrix-unit kernels). On
// gfx950 the product is a bf16 MFMA (v_mfma_f32_32x32x16_bf16); the packed
// Q8 / Q4 weights are read from HBM with 16-byte loads, dequantised in
// registers (value * fp16 block scale, rounded to bf16) and staged in LDS so
// every wave of the workgroup reuses them. Activations are staged in LDS too.
// LDS is double-buffered so one barrier per 64-wide K step suffices.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qg {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kQ8 = 0;
constexpr int kQ4 = 1;
constexpr int kBK = 64;              // K elements per pipeline step (two 32-element scale blocks)
constexpr int kRowBytes = kBK * 2;   // one bf16 tile row in LDS: 128 bytes = 8 chunks of 16 bytes
constexpr int kMaxExpertsPerLaunch = 128;

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

// Byte offset of 16-byte chunk `c` (0..7) of row `r` in a [rows][64] bf16 LDS tile.
// Chunks are XOR-swizzled by the row so that 32 lanes reading the same chunk
// column of 32 consecutive rows spread over all LDS banks.
__device__ __forceinline__ int lds_chunk(int r, int c) {
  return r * kRowBytes + ((c ^ (r & 7)) << 4);
}

// 16 int8 weights (one 16-byte load) -> 16 bf16 = w * s, as 8 packed dwords.
__device__ __forceinline__ void dequant_q8x16(const uint4 w, float s, uint32_t out[8]) {
  const uint32_t d[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float f0 = (float)(int8_t)(d[i]);
    const float f1 = (float)(int8_t)(d[i] >> 8);
    const float f2 = (float)(int8_t)(d[i] >> 16);
    const float f3 = (float)(int8_t)(d[i] >> 24);
    out[2 * i] = pack_bf16x2(f0 * s, f1 * s);
    out[2 * i + 1] = pack_bf16x2(f2 * s, f3 * s);
  }
}

// 32 packed nibbles (one 16-byte load, one scale block) -> 32 bf16 = (u - 8) * s,
// element 2j from the low nibble of byte j, element 2j+1 from its high nibble.
__device__ __forceinline__ void dequant_q4x32(const uint4 w, float s, uint32_t out[16]) {
  const uint32_t d[4] = {w.x, w.y, w.z, w.w};
  const float o = -8.0f * s;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const float lo = (float)((d[i] >> (8 * b)) & 0xFu);
      const float hi = (float)((d[i] >> (8 * b + 4)) & 0xFu);
      out[4 * i + b] = pack_bf16x2(__builtin_fmaf(lo, s, o), __builtin_fmaf(hi, s, o));
    }
  }
}

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
};

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

template <int FMT, int BM, int BN, int WM, int WN, bool MOE>
struct TileKernel {
  static constexpr int kThreads = WM * WN * 64;
  static constexpr int kWTM = BM / WM;        // rows per wave
  static constexpr int kWTN = BN / WN;        // cols per wave
  static constexpr int kTM = kWTM / 32;       // 32x32 MFMA blocks per wave (M)
  static constexpr int kTN = kWTN / 32;       // (N)
  static constexpr int kXChunks = BM * 8 / kThreads;            // 16-byte x chunks per thread per K step
  static constexpr int kWChunkElems = (FMT == kQ8) ? 16 : 32;   // weights per 16-byte load
  static constexpr int kWChunksPerRow = kBK / kWChunkElems;     // 4 (Q8) or 2 (Q4)
  static constexpr int kWChunks = BN * kWChunksPerRow / kThreads;
  static constexpr int kTileBytes = (BM + BN) * kRowBytes;
  static constexpr int kLdsBytes = 2 * kTileBytes;
  static_assert(kXChunks * kThreads == BM * 8, "x tile must split evenly");
  static_assert(kWChunks * kThreads == BN * kWChunksPerRow, "w tile must split evenly");
  static_assert(kTM >= 1 && kTN >= 1, "wave tile must hold a 32x32 block");
};

template <int FMT, int BM, int BN, int WM, int WN, bool MOE>
__device__ __forceinline__ void tile_body(const TileArgs& a, const uint8_t* __restrict__ wq,
                                          const uint16_t* __restrict__ sc, int m0, int n0,
                                          int rows_valid, const int* __restrict__ s_xrow,
                                          const int* __restrict__ s_yrow, char* __restrict__ lds) {
  using KT = TileKernel<FMT, BM, BN, WM, WN, MOE>;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN;
  const int wn = wave % WN;
  const int K = a.K;
  const int N = a.N;
  const int nk = (K + kBK - 1) / kBK;
  const int kblocks = K >> 5;
  const size_t wrow_bytes = (FMT == kQ8) ? (size_t)K : (size_t)(K >> 1);

  // --- per-thread x rows (fixed across the K loop) ---
  const uint16_t* xrow[KT::kXChunks];
  int xc[KT::kXChunks];
#pragma unroll
  for (int i = 0; i < KT::kXChunks; ++i) {
    const int q = tid + i * KT::kThreads;
    const int r = q >> 3;
    xc[i] = q & 7;
    int src = -1;
    if (r < rows_valid) src = MOE ? s_xrow[r] : (m0 + r);
    xrow[i] = (src >= 0) ? a.x + (size_t)src * K : nullptr;
  }
  // --- per-thread weight rows ---
  const uint8_t* wrow[KT::kWChunks];
  const uint16_t* srow[KT::kWChunks];
  int wc[KT::kWChunks];
#pragma unroll
  for (int i = 0; i < KT::kWChunks; ++i) {
    const int q = tid + i * KT::kThreads;
    const int r = q / KT::kWChunksPerRow;
    wc[i] = q % KT::kWChunksPerRow;
    const int n = n0 + r;
    wrow[i] = (n < N) ? wq + (size_t)n * wrow_bytes : nullptr;
    srow[i] = (n < N) ? sc + (size_t)n * kblocks : nullptr;
  }

  uint4 xr[KT::kXChunks];
  uint4 wr[KT::kWChunks];
  float sr[KT::kWChunks];

  auto load_step = [&](int kt) {
    const int k0 = kt * kBK;
#pragma unroll
    for (int i = 0; i < KT::kXChunks; ++i) {
      const int k = k0 + xc[i] * 8;
      if (xrow[i] != nullptr && k < K)
        xr[i] = *reinterpret_cast<const uint4*>(xrow[i] + k);
      else
        xr[i] = make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int i = 0; i < KT::kWChunks; ++i) {
      const int k = k0 + wc[i] * KT::kWChunkElems;
      if (wrow[i] != nullptr && k < K) {
        const size_t boff = (FMT == kQ8) ? (size_t)k : (size_t)(k >> 1);
        wr[i] = *reinterpret_cast<const uint4*>(wrow[i] + boff);
        sr[i] = fp16_to_f32(srow[i][k >> 5]);
      } else {
        wr[i] = make_uint4(0u, 0u, 0u, 0u);
        sr[i] = 0.0f;
      }
    }
  };

  auto store_step = [&](int buf) {
    char* xs = lds + buf * KT::kTileBytes;
    char* ws = xs + BM * kRowBytes;
#pragma unroll
    for (int i = 0; i < KT::kXChunks; ++i) {
      const int q = tid + i * KT::kThreads;
      *reinterpret_cast<uint4*>(xs + lds_chunk(q >> 3, q & 7)) = xr[i];
    }
#pragma unroll
    for (int i = 0; i < KT::kWChunks; ++i) {
      const int q = tid + i * KT::kThreads;
      const int r = q / KT::kWChunksPerRow;
      if constexpr (FMT == kQ8) {
        uint32_t o[8];
        dequant_q8x16(wr[i], sr[i], o);
        const int c = wc[i] * 2;
        *reinterpret_cast<uint4*>(ws + lds_chunk(r, c)) = make_uint4(o[0], o[1], o[2], o[3]);
        *reinterpret_cast<uint4*>(ws + lds_chunk(r, c + 1)) = make_uint4(o[4], o[5], o[6], o[7]);
      } else {
        uint32_t o[16];
        dequant_q4x32(wr[i], sr[i], o);
        const int c = wc[i] * 4;
#pragma unroll
        for (int h = 0; h < 4; ++h)
          *reinterpret_cast<uint4*>(ws + lds_chunk(r, c + h)) =
              make_uint4(o[4 * h], o[4 * h + 1], o[4 * h + 2], o[4 * h + 3]);
      }
    }
  };

  f32x16 acc[KT::kTM][KT::kTN];
#pragma unroll
  for (int i = 0; i < KT::kTM; ++i)
#pragma unroll
    for (int j = 0; j < KT::kTN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // 32-row MFMA blocks of this wave that hold at least one valid row
  const int wrow0 = wm * KT::kWTM;
  const int mblocks = rows_valid <= wrow0 ? 0 : (rows_valid - wrow0 + 31) >> 5;

  load_step(0);
  store_step(0);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = (kt + 1) < nk;
    if (more) load_step(kt + 1);

    const char* xs = lds + cur * KT::kTileBytes;
    const char* ws = xs + BM * kRowBytes;
    const int lr = lane & 31;
    const int lh = lane >> 5;
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const int c = kk * 2 + lh;
      bf16x8 bv[KT::kTN];
#pragma unroll
      for (int j = 0; j < KT::kTN; ++j)
        bv[j] = *reinterpret_cast<const bf16x8*>(ws + lds_chunk(wn * KT::kWTN + j * 32 + lr, c));
#pragma unroll
      for (int i = 0; i < KT::kTM; ++i) {
        if (i < mblocks) {
          const bf16x8 av = *reinterpret_cast<const bf16x8*>(xs + lds_chunk(wrow0 + i * 32 + lr, c));
#pragma unroll
          for (int j = 0; j < KT::kTN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv[j], acc[i][j], 0, 0, 0);
        }
      }
    }

    if (more) store_step(cur ^ 1);
    __syncthreads();
  }

  // --- epilogue: lane holds column (lane & 31) and rows (r/4)*8 + (lane/32)*4 + r%4 of each block ---
  const int lr = lane & 31;
  const int lh = lane >> 5;
#pragma unroll
  for (int i = 0; i < KT::kTM; ++i) {
    if (i >= mblocks) continue;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = wrow0 + i * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
      if (row >= rows_valid) continue;
      const int dst = MOE ? s_yrow[row] : (m0 + row);
      if (dst < 0) continue;
      float* yrow = a.y + (size_t)dst * N;
#pragma unroll
      for (int j = 0; j < KT::kTN; ++j) {
        const int col = n0 + wn * KT::kWTN + j * 32 + lr;
        if (col < N) yrow[col] = acc[i][j][r];
      }
    }
  }
}

template <int FMT, int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(WM * WN * 64) void dense_kernel(TileArgs a, const uint8_t* __restrict__ wq,
                                                             const uint16_t* __restrict__ sc) {
  using KT = TileKernel<FMT, BM, BN, WM, WN, false>;
  __shared__ __attribute__((aligned(16))) char lds[KT::kLdsBytes];
  const int mt_n = (a.M + BM - 1) / BM;
  const int nt_n = (a.N + BN - 1) / BN;
  const int ntiles = mt_n * nt_n;
  const int tile = xcd_tile(blockIdx.x, ntiles);
  // column-tile major: consecutive tiles (same XCD) share a weight column tile
  const int nt = tile / mt_n;
  const int mt = tile - nt * mt_n;
  const int m0 = mt * BM;
  const int rows_valid = min(BM, a.M - m0);
  tile_body<FMT, BM, BN, WM, WN, false>(a, wq, sc, m0, nt * BN, rows_valid, nullptr, nullptr, lds);
}

// Grouped MoE GEMM: the launch covers experts [e_begin, e_begin + n_experts).
// Work items are (expert, m tile, n tile) over active experts only; every
// workgroup decodes its item from the per-expert counts, so the host never
// needs the routing.
template <int FMT, int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(WM * WN * 64) void moe_kernel(TileArgs a, ExpertPtrs ep) {
  using KT = TileKernel<FMT, BM, BN, WM, WN, true>;
  __shared__ __attribute__((aligned(16))) char lds[KT::kLdsBytes];
  __shared__ int s_prefix[kMaxExpertsPerLaunch + 1];
  __shared__ int s_rowidx[BM];   // y row (assignment) of each tile row
  __shared__ int s_xrow[BM];     // x row (token = assignment / topk) of each tile row
  const int tid = threadIdx.x;
  const int nt_n = (a.N + BN - 1) / BN;
  const int ne = a.n_experts;

  // per-expert tile counts -> inclusive prefix (one thread; at most 128 experts)
  if (tid == 0) {
    int run = 0;
    s_prefix[0] = 0;
    for (int e = 0; e < ne; ++e) {
      const int lo = a.offsets[a.e_begin + e];
      const int hi = a.offsets[a.e_begin + e + 1];
      int c = hi - lo;
      if (lo < 0 || hi > a.M || c < 0) c = 0;   // inconsistent table: no work for this expert
      run += ((c + BM - 1) / BM) * nt_n;
      s_prefix[e + 1] = run;
    }
  }
  __syncthreads();
  const int ntiles = s_prefix[ne];
  if ((int)blockIdx.x >= ntiles) return;
  const int tile = xcd_tile(blockIdx.x, ntiles);
  // largest e with s_prefix[e] <= tile
  int lo = 0, hi = ne;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (s_prefix[mid] <= tile) lo = mid; else hi = mid;
  }
  const int e = lo;
  const int local = tile - s_prefix[e];
  const int mt = local / nt_n;           // m-tile major: consecutive tiles share the gathered rows
  const int nt = local - mt * nt_n;
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
  tile_body<FMT, BM, BN, WM, WN, true>(a, ep.wq[e], ep.sc[e], 0, nt * BN, rows_valid, s_xrow, s_rowidx, lds);
}

}  // namespace qg
