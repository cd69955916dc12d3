// Small-M dense GEMM (at most 16 activation rows, or up to 128 in blocks of 16): the shape of
// decode and of batched speculative-draft verification, which the paper names as the
// memory-bound side of inference (Section 2.3) and as future work for its matrix-unit kernels
// (Section 5.2), and of short prompts whose few output tiles would leave most CUs idle. Every packed weight
// is read once and the arithmetic per weight byte is tiny, so the call is bound by HBM bandwidth:
// there is no LDS staging of the weights. Each lane dequantises its own 16-byte weight load
// straight into MFMA operand registers (v_mfma_f32_16x16x32_bf16, weights as the 16-row A
// operand, activations as the 16-column B operand, columns past M fed with zeros).
//
// Work split: a workgroup of WAVES waves owns 32 weight rows and a contiguous range of K chunks;
// wave w takes every WAVES-th chunk of that range, w first. A chunk is the 64 bytes of a weight
// row that one lane group of a load instruction covers: 64 K elements for Q8 (lane group g
// loads elements 16g..16g+15) and 128 for Q4 (lane group g loads the 32-element block g). A wave
// keeps kSmDepth<FMT> chunks in flight and issues the next chunk's loads as soon as it has dequantised
// one: with every chunk issued up front, the memory system would return the chunks of all
// waves in no particular order, leaving many waves idle until late and piling the
// dequantisation up at the end.
// The block scales of the workgroup's rows and K range are read with consecutive lanes on
// consecutive scales (a few cache lines per load instead of one line per row) and handed to
// the lanes that use them through LDS.
// Partial sums are combined in a fixed order: chunks in increasing order inside a wave, waves
// 0..WAVES-1 through LDS (each output piece added up by one wave), then (when K is split over
// workgroups) splits 0..S-1 by a second kernel.
// Results are therefore bitwise reproducible.
#pragma once

#include "qgemm_kernels.hpp"

namespace qg {

constexpr int kSmRows = 32;       // weight rows per workgroup: two 16-row MFMA groups per wave
constexpr int kSmMaxM = 16;       // activation rows of one MFMA B operand (16 columns)
constexpr int kSmMaxMT = 8;       // 16-column activation blocks per call at most (M <= 128)
constexpr int kSmWaves = 8;       // waves per workgroup
// chunks of a wave in flight: three for Q8, two for Q4, whose four dequantisation units per
// load make the VALU work of a chunk twice as long (measured on MI355X at M = 1, 4, 16: Q8 three
// 0-5% faster than two, Q4 three 8-15% slower; four, or 16 waves of two chunks, slower for both)
template <int FMT>
constexpr int kSmDepth = (FMT == kQ8) ? 3 : 2;

struct SmallArgs {
  const uint16_t* x;      // bf16 [M][K]
  const uint8_t* wq;      // packed weights [N][row bytes]
  const uint16_t* sc;     // fp16 scales [N][K / 32]
  float* y;               // fp32 [M][N]
  int M;
  int N;
  int K;
  int splits;             // workgroups along K per 32-row block
  int cps;                // chunks per split (the last split may hold fewer)
  int nbp_log2;           // log2 of the scale blocks staged per row (a power of two >= cps * blocks per chunk)
  float* ws;              // [splits][M][N] fp32 partials, used when splits > 1
};

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

template <int FMT>
struct SmallFmt {
  static constexpr int kKC = (FMT == kQ8) ? 64 : 128;   // K elements per chunk
  static constexpr int kU = (FMT == kQ8) ? 2 : 4;       // 8-element MFMA units per 16-byte weight load
  static constexpr int kBPC = kKC / 32;                 // scale blocks per chunk
};

// LDS bytes of the staged scales: 32 rows of (2^nbp_log2 + 2) fp16 (the 2 shift consecutive
// rows by one LDS bank).
__host__ __device__ constexpr int smallm_scale_lds_bytes(int nbp_log2) {
  return kSmRows * ((1 << nbp_log2) + 2) * 2;
}

// JW: chunks per wave held in registers (the host keeps ceil(cps / WAVES) <= JW and
// cps * blocks per chunk <= 2^nbp_log2 <= JW * WAVES * blocks per chunk).
// MT: 16-column blocks of activation rows (M <= 16 MT): every dequantised weight operand feeds
// MT MFMAs, one per block, so a weight is still read and dequantised once per call.
template <int FMT, int JW, int WAVES, int MT = 1>
__global__ __launch_bounds__(WAVES * 64) void smallm_kernel(SmallArgs a) {
  using F = SmallFmt<FMT>;
  constexpr int KC = F::kKC;
  constexpr int U = F::kU;
  constexpr int EPL = 8 * U;                           // K elements per lane per chunk
  constexpr int T = WAVES * 64;
  constexpr int SL = (kSmRows * JW * WAVES * F::kBPC + T - 1) / T;   // scale loads per thread (upper bound)
  extern __shared__ uint16_t s_scale[];
  __shared__ f32x4 red[WAVES][2 * MT][64];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int r16 = lane & 15;
  const int g = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;
  const int p = blockIdx.x / a.splits;
  const int s = blockIdx.x - p * a.splits;
  const int n0 = p * kSmRows;
  const int nc = (K + KC - 1) / KC;
  const int c_begin = s * a.cps;
  const int c_end = min(nc, c_begin + a.cps);
  const uint32_t rowbytes = (FMT == kQ8) ? (uint32_t)K : (uint32_t)K / 2u;
  const int nblk = K / 32;
  const int blk0 = c_begin * F::kBPC;
  const int nbp_log2 = a.nbp_log2;
  const int sstride = (1 << nbp_log2) + 2;

  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.wq, (uint32_t)N * rowbytes);
  const __amdgpu_buffer_rsrc_t sr = make_rsrc(a.sc, (uint32_t)N * (uint32_t)nblk * 2u);
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, (uint32_t)M * (uint32_t)K * 2u);

  // scales of rows n0..n0+31, blocks blk0..blk0+2^nbp_log2-1, row-major over the threads
  uint32_t sv[SL];
#pragma unroll
  for (int q = 0; q < SL; ++q) {
    const int idx = tid + q * T;
    const int row = idx >> nbp_log2;
    const int blk = idx & ((1 << nbp_log2) - 1);
    const bool live = row < kSmRows && n0 + row < N && blk0 + blk < nblk;
    const uint32_t so = live ? ((uint32_t)(n0 + row) * (uint32_t)nblk + (uint32_t)(blk0 + blk)) * 2u : kOOB;
    sv[q] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(sr, so, 0, 0);
  }
  // weights and activations, chunk by chunk, at most kSmDepth chunks of a wave in flight (fewer
  // with several activation blocks, whose loads take MT times the registers)
  uint4 w[JW][2];
  u32x4 xv[JW][MT][U];
  auto issue = [&](int j) {
    const int c = c_begin + wave + WAVES * j;
    const int kst = c * KC + g * EPL;          // first K element of this lane's load
    const bool ok = c < c_end && kst < K;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int n = n0 + 16 * i + r16;
      const bool live = ok && n < N;
      const uint32_t wo = live ? (uint32_t)n * rowbytes + (uint32_t)c * 64u + (uint32_t)g * 16u : kOOB;
      w[j][i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(wr, wo, 0, 0));
    }
#pragma unroll
    for (int cb = 0; cb < MT; ++cb) {
      const int m = 16 * cb + r16;
      const bool xok = ok && m < M;
      const uint32_t xo = ((uint32_t)m * (uint32_t)K + (uint32_t)kst) * 2u;
#pragma unroll
      for (int u = 0; u < U; ++u)
        xv[j][cb][u] =
            __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, xok ? xo + 16u * u : kOOB, 0, 0));
    }
  };
  constexpr int kDepth = MT == 1 ? kSmDepth<FMT> : (MT == 2 ? 2 : 1);
  constexpr int D = JW < kDepth ? JW : kDepth;
#pragma unroll
  for (int j = 0; j < D; ++j) issue(j);
  __builtin_amdgcn_sched_barrier(0);   // keep these loads ahead of the first LDS write
#pragma unroll
  for (int q = 0; q < SL; ++q) {
    const int idx = tid + q * T;
    const int row = idx >> nbp_log2;
    if (row < kSmRows) s_scale[row * sstride + (idx & ((1 << nbp_log2) - 1))] = (uint16_t)sv[q];
  }
  __syncthreads();

  f32x4 acc[2][MT];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int cb = 0; cb < MT; ++cb) acc[i][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < JW; ++j) {
    const int c = c_begin + wave + WAVES * j;
    const bool ok = c < c_end && c * KC + g * EPL < K;
    const int bl = (c - c_begin) * F::kBPC + ((FMT == kQ8) ? (g >> 1) : g);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      // a masked chunk has zero weight bytes and takes a zero scale, so its weights are all zero
      const uint16_t sh = s_scale[ok ? (16 * i + r16) * sstride + bl : 0];
      const float sf = ok ? fp16_to_f32(sh) : 0.0f;
      const uint4 d = w[j][i];
      u32x4 wu[U];
      if constexpr (FMT == kQ8) {
        wu[0] = dequant_q8_unit(d.x, d.y, sf);
        wu[1] = dequant_q8_unit(d.z, d.w, sf);
      } else {
        float s24, s20, off;
        q4_factors(sf, s24, s20, off);
        wu[0] = dequant_q4_unit(d.x, s24, s20, off);
        wu[1] = dequant_q4_unit(d.y, s24, s20, off);
        wu[2] = dequant_q4_unit(d.z, s24, s20, off);
        wu[3] = dequant_q4_unit(d.w, s24, s20, off);
      }
#pragma unroll
      for (int cb = 0; cb < MT; ++cb)
#pragma unroll
        for (int u = 0; u < U; ++u)
          acc[i][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wu[u]),
                                                              __builtin_bit_cast(bf16x8_t, xv[j][cb][u]), acc[i][cb],
                                                              0, 0, 0);
    }
    if (j + D < JW) {
      __builtin_amdgcn_sched_barrier(0);
      issue(j + D);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // every wave hands its sums over through LDS; piece b (row group b / MT, column block b % MT) is
  // then added by wave b % WAVES in wave order 0 .. WAVES-1 and stored by it
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int cb = 0; cb < MT; ++cb) red[wave][i * MT + cb][lane] = acc[i][cb];
  __syncthreads();

  // lane holds output column m = 16 cb + r16 (activation row) and weight rows nb..nb+3 of its
  // piece; with K split over workgroups the partial goes to ws[s] and a second kernel sums the
  // splits
  const bool vec = (N & 3) == 0;
#pragma unroll
  for (int b0 = 0; b0 < 2 * MT; b0 += WAVES) {
    const int b = b0 + wave;
    if (b >= 2 * MT) break;
    f32x4 sum = red[0][b][lane];
#pragma unroll
    for (int v = 1; v < WAVES; ++v) sum += red[v][b][lane];
    const int i = b / MT, cb = b % MT;
    const int m = 16 * cb + r16;
    if (m >= M) continue;
    float* dst = (a.splits == 1) ? a.y + (size_t)m * N : a.ws + ((size_t)s * M + m) * N;
    const int nb = n0 + 16 * i + 4 * g;
    if (vec && nb + 3 < N) {
      *reinterpret_cast<f32x4*>(dst + nb) = sum;
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (nb + r < N) dst[nb + r] = sum[r];
    }
  }
}

// y[e] = sum_{s < splits} ws[s][e] over `total` elements, in increasing s (deterministic).
__global__ __launch_bounds__(256) void smallm_reduce_kernel(const float* __restrict__ ws, float* __restrict__ y,
                                                            long total, int splits) {
  const long e0 = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (e0 >= total) return;
  if (e0 + 4 <= total && (total & 3) == 0) {
    f32x4 acc = *reinterpret_cast<const f32x4*>(ws + e0);
    for (int s = 1; s < splits; ++s) acc += *reinterpret_cast<const f32x4*>(ws + (long)s * total + e0);
    *reinterpret_cast<f32x4*>(y + e0) = acc;
  } else {
    for (long e = e0; e < e0 + 4 && e < total; ++e) {
      float acc = ws[e];
      for (int s = 1; s < splits; ++s) acc += ws[(long)s * total + e];
      y[e] = acc;
    }
  }
}

}  // namespace qg
