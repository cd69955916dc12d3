// Bandwidth-bound helpers around the grouped GEMM: stable bucketing of token
// slots by expert (each active expert needs the list of tokens routed to it,
// Section 3.1 MoE expert GEMM item), the SiLU-gated activation between the
// gate/up and down projections (Section 3.1, fused gate/up item) and the
// router-weighted combine of the selected experts' outputs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qg {

constexpr int kBucketThreads = 256;
constexpr int kBadExpert = INT32_MIN;

// Per-block histogram of expert ids over a chunk of `chunk` assignments.
// counts: [gridDim.x][E]
__global__ __launch_bounds__(kBucketThreads) void bucket_count_kernel(const int32_t* __restrict__ idx, int n,
                                                                      int E, int chunk,
                                                                      int32_t* __restrict__ counts) {
  extern __shared__ int32_t hist[];
  for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = 0;
  __syncthreads();
  const long base = (long)blockIdx.x * chunk;
  for (int i = threadIdx.x; i < chunk; i += blockDim.x) {
    const long a = base + i;
    if (a >= n) break;
    const int e = idx[a];
    if (e >= 0 && e < E) atomicAdd(&hist[e], 1);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) counts[(long)blockIdx.x * E + e] = hist[e];
}

// Stable scatter: perm[offsets[e] + r] = the r-th assignment (in increasing
// order) routed to expert e. Each block places its chunk after the entries of
// earlier blocks (prefix of `counts`), then walks the chunk in rounds of
// blockDim assignments; inside a round, lanes with equal expert ids are
// ranked by lane order (wave ballots) and waves are taken in order.
// An expert whose total count disagrees with offsets (or whose segment leaves
// [0, n)) is marked bad: its declared segment is filled with -1, its
// assignments are skipped, the error flag receives `seq`, and if `ypoison` is
// given the y rows of those assignments (and of out-of-range ids) become NaN.
__global__ __launch_bounds__(kBucketThreads) void bucket_scatter_kernel(
    const int32_t* __restrict__ idx, const int32_t* __restrict__ offsets, int n, int E, int chunk,
    const int32_t* __restrict__ counts, int nblk, int32_t* __restrict__ perm, int32_t* __restrict__ err_flag,
    int seq, float* __restrict__ ypoison, int N) {
  extern __shared__ int32_t cursor[];
  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += blockDim.x) {
    const int lo = offsets[e];
    const int hi = offsets[e + 1];
    long c = lo;
    long tot = 0;
#pragma unroll 16
    for (int b = 0; b < nblk; ++b) {
      const int v = counts[(long)b * E + e];
      if (b < (int)blockIdx.x) c += v;
      tot += v;
    }
    const bool bad = (lo < 0) || (hi > n) || (hi < lo) || (tot != (long)hi - lo) || (e == 0 && lo != 0);
    cursor[e] = bad ? kBadExpert : (int)c;
    if (bad) {
      if (blockIdx.x == 0) {
        err_flag[0] = seq;
        const int s0 = lo < 0 ? 0 : lo;
        const int s1 = hi > n ? n : hi;
        for (int p = s0; p < s1; ++p) perm[p] = -1;
      }
    }
  }
  __syncthreads();

  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int nwaves = blockDim.x >> 6;
  int nbits = 0;
  while ((1 << nbits) < E) ++nbits;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const long base = (long)blockIdx.x * chunk;
  for (int r0 = 0; r0 < chunk; r0 += blockDim.x) {
    const long a = base + r0 + tid;
    const bool valid = (r0 + tid < chunk) && (a < n);
    const int e = valid ? idx[a] : -1;
    const bool inrange = valid && e >= 0 && e < E;
    if (valid && !inrange) {
      err_flag[0] = seq;
      if (ypoison != nullptr)
        for (int j = 0; j < N; ++j) ypoison[a * (long)N + j] = __builtin_nanf("");
    }
    uint64_t same = __ballot(inrange);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = inrange && ((e >> b) & 1);
      const uint64_t m = __ballot(bit);
      same &= bit ? m : ~m;
    }
    const int rank = __popcll(same & lt_mask);
    const int cnt = __popcll(same);
    for (int w = 0; w < nwaves; ++w) {
      if (wave == w && inrange) {
        const int cb = cursor[e];
        if (cb != kBadExpert) {
          perm[cb + rank] = (int32_t)a;
        } else if (ypoison != nullptr) {
          for (int j = 0; j < N; ++j) ypoison[a * (long)N + j] = __builtin_nanf("");
        }
        if (rank == 0 && cb != kBadExpert) cursor[e] = cb + cnt;
      }
      __syncthreads();
    }
  }
}

// h[r][i] = bf16(silu(g) * u), g = y1[r][i], u = y1[r][inter + i]; 8 outputs per thread.
__global__ __launch_bounds__(256) void swiglu_kernel(const float* __restrict__ y1, uint16_t* __restrict__ h,
                                                     long groups, int inter) {
  const long gid = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= groups) return;
  const int per_row = inter >> 3;
  const long r = gid / per_row;
  const int i0 = (int)(gid - r * per_row) * 8;
  const float* grow = y1 + r * (2L * inter) + i0;
  const float4 g0 = *reinterpret_cast<const float4*>(grow);
  const float4 g1 = *reinterpret_cast<const float4*>(grow + 4);
  const float4 u0 = *reinterpret_cast<const float4*>(grow + inter);
  const float4 u1 = *reinterpret_cast<const float4*>(grow + inter + 4);
  const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
  const float u[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float a0 = swiglu_f32(g[2 * i], u[2 * i]);
    const float a1 = swiglu_f32(g[2 * i + 1], u[2 * i + 1]);
    o[i] = pack_bf16x2(a0, a1);
  }
  *reinterpret_cast<uint4*>(h + r * inter + i0) = make_uint4(o[0], o[1], o[2], o[3]);
}

// out[t][n] = sum_j w[t*topk+j] * y2[t*topk+j][n], fp32 fused multiply-add in increasing j.
// Each thread produces V (4 or 8) outputs of one token row as V/4 groups of 4 consecutive ones,
// keeping V/4 * topk independent 16-byte loads in flight. With SPREAD thread i of the row takes
// 4-float chunks i, i + N/V, ..., so every wave-wide load or store covers 1 KiB of contiguous
// memory (faster when y2 is still in the last-level cache); otherwise its V outputs are
// consecutive (faster when y2 streams from HBM). y2 is read exactly once, so its loads and the
// output stores are non-temporal.
template <int V, int KFIX, bool SPREAD>
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ y2, const float* __restrict__ w,
                                                      float* __restrict__ out, long groups, int topk_rt, int N) {
  static_assert(V == 4 || V == 8, "4 or 8 outputs per thread");
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  constexpr int G = V / 4;
  const int topk = KFIX > 0 ? KFIX : topk_rt;
  const long gid = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= groups) return;
  const int per_row = N / V;
  const long t = gid / per_row;
  const int i = (int)(gid - t * per_row);
  int ncol[G];   // first column of each group of 4
#pragma unroll
  for (int g = 0; g < G; ++g) ncol[g] = SPREAD ? 4 * (i + g * per_row) : V * i + 4 * g;
  f32x4 acc[G];
#pragma unroll
  for (int g = 0; g < G; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
  if constexpr (KFIX > 0) {
    // every slot's loads first, then the FMAs in slot order
    f32x4 v[KFIX][G];
    float wj[KFIX];
#pragma unroll
    for (int j = 0; j < KFIX; ++j) {
      const long a = t * KFIX + j;
      wj[j] = w[a];
#pragma unroll
      for (int g = 0; g < G; ++g) v[j][g] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(y2 + a * N + ncol[g]));
    }
#pragma unroll
    for (int j = 0; j < KFIX; ++j)
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[g][c] = __builtin_fmaf(wj[j], v[j][g][c], acc[g][c]);
  } else {
    for (int j = 0; j < topk; ++j) {
      const long a = t * topk + j;
      const float wj = w[a];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(y2 + a * N + ncol[g]));
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[g][c] = __builtin_fmaf(wj, v[c], acc[g][c]);
      }
    }
  }
#pragma unroll
  for (int g = 0; g < G; ++g) __builtin_nontemporal_store(acc[g], reinterpret_cast<f32x4*>(out + t * N + ncol[g]));
}

// p[i] = v for i < n, four entries per thread (clears counters without a memset node).
__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t* __restrict__ p, long n, int v) {
  const long i0 = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
#pragma unroll
  for (int k = 0; k < 4; ++k)
    if (i0 + k < n) p[i0 + k] = v;
}

// y[i] = sum_{s < splits} ws[s][i], summed in increasing s (deterministic); 4 floats per thread.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ ws, float* __restrict__ y,
                                                            long n4, int splits, long stride) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  float4 acc = reinterpret_cast<const float4*>(ws)[i];
  for (int s = 1; s < splits; ++s) {
    const float4 v = reinterpret_cast<const float4*>(ws + (long)s * stride)[i];
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  reinterpret_cast<float4*>(y)[i] = acc;
}

}  // namespace qg

namespace qg {

// Measurement probe (not on the GEMM path): every wave issues `iters` rounds of four independent
// bf16 MFMAs (v_mfma_f32_32x32x16_bf16, the GEMM's instruction) on register operands, so the
// matrix cores run at their sustained rate. Wave 0 of each workgroup records the shader-clock
// counter and the constant-rate real-time counter before and after; their ratio is the clock the
// chip holds under full matrix-core load. out: [gridDim.x][4] int64 (clock start, clock end,
// real-time start, real-time end); sink keeps the accumulators alive (written only if a lane's sum
// is exactly 1234.5, which the operands never produce).
constexpr int kProbeThreads = 512;
__global__ __launch_bounds__(kProbeThreads) void mfma_clock_probe_kernel(long long* __restrict__ out, int iters,
                                                                          float* __restrict__ sink) {
  // 96 KiB of LDS: at most one workgroup per CU (160 KiB), so a grid of one workgroup per CU
  // puts eight waves, two per SIMD, on every CU at once
  __shared__ char probe_lds[96 * 1024];
  typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
  typedef float f32x16_t __attribute__((ext_vector_type(16)));
  const int lane = threadIdx.x & 63;
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)((lane + i) & 7));
    b[i] = (__bf16)(0.002f * (float)((lane * 3 + i) & 7));
  }
  f32x16_t c0 = {}, c1 = {}, c2 = {}, c3 = {};
  __syncthreads();
  long long t0 = 0, r0 = 0;
  if (threadIdx.x == 0) {
    t0 = (long long)__builtin_readcyclecounter();
    r0 = (long long)__builtin_amdgcn_s_memrealtime();
  }
  for (int it = 0; it < iters; ++it) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  if (s == 1234.5f) sink[threadIdx.x] = s + (float)probe_lds[threadIdx.x];
  __syncthreads();
  if (threadIdx.x == 0) {
    const long long t1 = (long long)__builtin_readcyclecounter();
    const long long r1 = (long long)__builtin_amdgcn_s_memrealtime();
    long long* o = out + 4 * (long)blockIdx.x;
    o[0] = t0;
    o[1] = t1;
    o[2] = r0;
    o[3] = r1;
  }
}

}  // namespace qg
