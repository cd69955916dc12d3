// C ABI of the block-quantised prefill GEMM library (declarations and the
// contract of every entry point are in include/qgemm.h).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/qgemm.h"
#include "qgemm_kernels.hpp"
#include "qgemm_aux.hpp"
#include "qgemm_smallm.hpp"
#include "attn_kernels.hpp"

// Scratch of qgemm_moe_noalloc (2 MiB + 256 bytes per device, held until the process ends): the
// token-slot permutation, the per-block expert histograms and the error flag. In host code this
// name is only a stand-in for the symbol; kernels get the per-device address from
// hipGetSymbolAddress.
static __device__ __align__(256) int32_t scratch[(1 << 18) + (1 << 18) + 64];

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int ok() {
  g_last_error.clear();
  return QGEMM_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(QGEMM_EHIP, "%s: kernel launch failed: %s", what, hipGetErrorString(e));
  return QGEMM_OK;
}

int check_common(int N, int K, int fmt) {
  if (fmt != QGEMM_Q8 && fmt != QGEMM_Q4) return fail(QGEMM_EINVAL, "unknown weight format %d", fmt);
  if (N < 1) return fail(QGEMM_EINVAL, "N must be >= 1 (got %d)", N);
  if (K < 32 || K % 32 != 0) return fail(QGEMM_EINVAL, "K must be a positive multiple of 32 (got %d)", K);
  return QGEMM_OK;
}

// ---------------------------------------------------------------------------
// kernel selection
// ---------------------------------------------------------------------------

template <int FMT, int BM, int BN, int WM, int WN, int XS>
int launch_dense(const qg::TileArgs& a, const void* wq, const void* sc, hipStream_t s) {
  const long tiles = (long)((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * a.splits;
  if (tiles > 0x7fffffffL) return fail(QGEMM_EUNSUPPORTED, "too many tiles");
  hipLaunchKernelGGL((qg::dense_kernel<FMT, BM, BN, WM, WN, XS>), dim3((unsigned)tiles), dim3(WM * WN * 64), 0, s, a,
                     static_cast<const uint8_t*>(wq), static_cast<const uint16_t*>(sc));
  return check_launch("qgemm_dense");
}

// split-K partials (per device; grown on first use, then reused)
std::mutex g_split_mutex;
std::vector<std::pair<float*, size_t>> g_split_ws;

int split_workspace(size_t floats, float** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return fail(QGEMM_EHIP, "hipGetDevice failed");
  }
  if ((int)g_split_ws.size() <= dev) g_split_ws.resize(dev + 1, {nullptr, 0});
  auto& w = g_split_ws[dev];
  if (w.second < floats) {
    if (w.first) (void)hipFree(w.first);   // waits for work that may still use it
    w = {nullptr, 0};
    if (hipMalloc(reinterpret_cast<void**>(&w.first), floats * sizeof(float)) != hipSuccess) {
      (void)hipGetLastError();
      return fail(QGEMM_EHIP, "hipMalloc of %zu bytes for split-K partials failed", floats * sizeof(float));
    }
    w.second = floats;
  }
  *out = w.first;
  return QGEMM_OK;
}

constexpr int kMinStepsPerSplit = 12;

constexpr long kSmTargetGroups = 256;   // workgroups (of eight waves) to fill the CUs without a K split
constexpr int kSmMaxJW = 8;             // chunks per wave held in registers

template <int FMT, int JW, int MT>
int launch_small(const qg::SmallArgs& a, long groups, hipStream_t s) {
  hipLaunchKernelGGL((qg::smallm_kernel<FMT, JW, qg::kSmWaves, MT>), dim3((unsigned)groups), dim3(qg::kSmWaves * 64),
                     qg::smallm_scale_lds_bytes(a.nbp_log2), s, a);
  return check_launch("qgemm_dense (small M)");
}

template <int FMT, int MT>
int launch_small_jw(const qg::SmallArgs& a, int JW, long groups, hipStream_t s) {
  switch (JW) {
    case 1: return launch_small<FMT, 1, MT>(a, groups, s);
    case 2: return launch_small<FMT, 2, MT>(a, groups, s);
    case 4: return launch_small<FMT, 4, MT>(a, groups, s);
    default: return launch_small<FMT, 8, MT>(a, groups, s);
  }
}

// M <= 16 (or up to 128 in MT blocks of 16 columns): 32 weight rows per workgroup; K is split
// over workgroups only when there are fewer than 256 row blocks (or a wave would hold more than
// kSmMaxJW chunks). With several column blocks the call is latency-bound rather than
// weight-streaming, and a split keeps at least 4 chunks per workgroup (measured on the split
// targets 32 / 64 / 128 / 256: 128x1024x1024 Q8 11.0 / 9.6 / 9.5 / 10.5 us, 128x2048x8192 Q8
// 38 / 38 / 38 / 24 us, 96x2048x768 Q4 9.2 / 9.2 / 10.3 / 10.4 us; this rule picks the best of
// each). Split partials go to the split-K workspace and a second kernel adds them in split order.
template <int FMT>
int small_dispatch(const qg::TileArgs& t, const void* wq, const void* sc, hipStream_t s) {
  using F = qg::SmallFmt<FMT>;
  const int MT = t.M <= 16 ? 1 : t.M <= 32 ? 2 : t.M <= 64 ? 4 : 8;
  const long nc = (t.K + F::kKC - 1) / F::kKC;
  const long P = (t.N + qg::kSmRows - 1) / qg::kSmRows;
  long S = std::min<long>(nc, (kSmTargetGroups + P - 1) / P);
  if (MT > 1) S = std::min<long>(S, std::max<long>(1, nc / 4));
  S = std::max<long>(S, (nc + qg::kSmWaves * kSmMaxJW - 1) / (qg::kSmWaves * kSmMaxJW));
  const long cps = (nc + S - 1) / S;
  S = (nc + cps - 1) / cps;
  if (P * S > 0x7fffffffL) return fail(QGEMM_EUNSUPPORTED, "too many workgroups");
  int JW = 1;
  while (JW * qg::kSmWaves < cps) JW *= 2;
  int nbp_log2 = 0;
  while ((1L << nbp_log2) < cps * F::kBPC) ++nbp_log2;
  qg::SmallArgs a{};
  a.x = t.x;
  a.wq = static_cast<const uint8_t*>(wq);
  a.sc = static_cast<const uint16_t*>(sc);
  a.y = t.y;
  a.M = t.M;
  a.N = t.N;
  a.K = t.K;
  a.splits = (int)S;
  a.cps = (int)cps;
  a.nbp_log2 = nbp_log2;
  std::unique_lock<std::mutex> lock(g_split_mutex, std::defer_lock);
  const long total = (long)t.M * t.N;
  if (S > 1) {
    lock.lock();
    int rc = split_workspace((size_t)S * total, &a.ws);
    if (rc != QGEMM_OK) return rc;
  }
  int rc;
  switch (MT) {
    case 1: rc = launch_small_jw<FMT, 1>(a, JW, P * S, s); break;
    case 2: rc = launch_small_jw<FMT, 2>(a, JW, P * S, s); break;
    case 4: rc = launch_small_jw<FMT, 4>(a, JW, P * S, s); break;
    default: rc = launch_small_jw<FMT, 8>(a, JW, P * S, s); break;
  }
  if (rc != QGEMM_OK || S == 1) return rc;
  hipLaunchKernelGGL(qg::smallm_reduce_kernel, dim3((unsigned)((total + 1023) / 1024)), dim3(256), 0, s, a.ws, a.y,
                     total, (int)S);
  return check_launch("qgemm_dense (small M) split reduction");
}

template <int FMT>
int dense_dispatch(qg::TileArgs a, const void* wq, const void* sc, hipStream_t s) {
  if (a.M <= qg::kSmMaxM) return small_dispatch<FMT>(a, wq, sc, s);
  // up to 128 rows, when the 128x128 tiles would occupy few CUs (each walking the whole K range
  // alone), the small-M kernel with MT blocks of 16 activation columns spreads K over waves; its
  // cost grows with MT, so it takes over while (128-wide column tiles) x MT <= 512 (measured:
  // 128x8192x2048 Q8 20.6 against 29.1 us with the tiles, 64x14336x4096 Q4 40 against 60 us,
  // 17x8192x2048 Q8 7.5 against 32.6 us; 128x16384x2048 Q8 39 against 31 us stays on the tiles)
  if (a.M <= qg::kSmMaxM * qg::kSmMaxMT) {
    const int MT = a.M <= 32 ? 2 : a.M <= 64 ? 4 : 8;
    if ((long)((a.N + 127) / 128) * MT <= 512) return small_dispatch<FMT>(a, wq, sc, s);
  }
  a.splits = 1;
  const long big = (long)((a.M + 255) / 256) * ((a.N + 255) / 256);
  if (a.M >= 256 && a.N >= 256 && big >= 200) return launch_dense<FMT, 256, 256, 2, 4, 2>(a, wq, sc, s);
  const int nk = (a.K + 63) / 64;
  // up to 1024 rows with few 256x256 tiles: 128x256 eight-wave tiles, twice the tiles, so half the
  // K split and half the fp32 partials; the split keeps tiles x splits <= 256 (one round). Up to
  // 2048 rows only where these tiles need no split. Measured against the 256x256 split: dense Q4
  // 512x8192x3072 48-49 vs 51-53 us, Q8 512x2048x2048 26.6 vs 34.4, Q4 768x1536x2048 27.0 vs 35.6,
  // Q8 256x8192x2048 29.2 vs 36.8, Q8 2048x4096x2048 49.6 vs 60.8, Q4 1536x4096x4096 78 vs 97 us;
  // Q8 2048x2048x8192 (two splits needed) 100 vs 92.7 us stays on the 256x256 split.
  const long t2 = (long)((a.M + 127) / 128) * ((a.N + 255) / 256);
  if (a.M >= 128 && a.N >= 256 && ((long)a.M * a.N) % 4 == 0 && (a.M <= 1024 || (a.M <= 2048 && t2 > 128))) {
    int S = (int)std::max<long>(1, std::min<long>(8, 256 / t2));
    while (S > 1 && nk / S < kMinStepsPerSplit) --S;
    if (S == 1) return launch_dense<FMT, 128, 256, 2, 4, 2>(a, wq, sc, s);
    const long mn = (long)a.M * a.N;
    std::lock_guard<std::mutex> lock(g_split_mutex);
    float* ws = nullptr;
    int rc = split_workspace((size_t)S * mn, &ws);
    if (rc != QGEMM_OK) return rc;
    a.ws = ws;
    a.splits = S;
    rc = launch_dense<FMT, 128, 256, 2, 4, 2>(a, wq, sc, s);
    if (rc != QGEMM_OK) return rc;
    const long n4 = mn / 4;
    hipLaunchKernelGGL(qg::splitk_reduce_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, ws, a.y, n4, S,
                       mn);
    return check_launch("qgemm_dense split-K reduction");
  }
  // few 256x256 tiles but a long K: split K over several workgroups per tile (fp32 partials,
  // summed in split order by a second kernel) so that every CU gets a 256x256 tile
  if (a.M >= 256 && a.N >= 256 && ((long)a.M * a.N) % 4 == 0) {
    int S = (int)std::min<long>(8, (256 + big - 1) / big);
    while (S > 1 && nk / S < kMinStepsPerSplit) --S;
    if (S > 1) {
      const long mn = (long)a.M * a.N;
      std::lock_guard<std::mutex> lock(g_split_mutex);
      float* ws = nullptr;
      int rc = split_workspace((size_t)S * mn, &ws);
      if (rc != QGEMM_OK) return rc;
      a.ws = ws;
      a.splits = S;
      rc = launch_dense<FMT, 256, 256, 2, 4, 2>(a, wq, sc, s);
      if (rc != QGEMM_OK) return rc;
      const long n4 = mn / 4;
      hipLaunchKernelGGL(qg::splitk_reduce_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, ws, a.y, n4, S,
                         mn);
      return check_launch("qgemm_dense split-K reduction");
    }
  }
  return launch_dense<FMT, 128, 128, 2, 2, 2>(a, wq, sc, s);
}

template <int FMT, int BM, int BN, int WM, int WN, int XS, bool SWI, bool CMB>
int launch_moe_cfg(qg::TileArgs a, const void* const* wq, const void* const* sc, int E, hipStream_t s) {
  const int nt = SWI ? (a.swi_inter + BN / 2 - 1) / (BN / 2) : (a.N + BN - 1) / BN;
  for (int e0 = 0; e0 < E; e0 += qg::kMaxExpertsPerLaunch) {
    const int ne = (E - e0) < qg::kMaxExpertsPerLaunch ? (E - e0) : qg::kMaxExpertsPerLaunch;
    qg::ExpertPtrs ep;
    for (int i = 0; i < qg::kMaxExpertsPerLaunch; ++i) {
      ep.wq[i] = i < ne ? static_cast<const uint8_t*>(wq[e0 + i]) : nullptr;
      ep.sc[i] = i < ne ? static_cast<const uint16_t*>(sc[e0 + i]) : nullptr;
    }
    a.e_begin = e0;
    a.n_experts = ne;
    // upper bound of sum_e ceil(c_e / BM) over the launch's experts (m-tile groups), rounded up
    // to whole runs on all 8 XCDs; workgroups past the real group count exit at once
    const long mt_bound = (long)(a.M + BM - 1) / BM + ne;
    constexpr long kDeal = 8L * qg::kMoeRun;   // groups per round over the 8 XCDs
    const long grid = (mt_bound + kDeal - 1) / kDeal * kDeal * nt;
    if (grid > 0x7fffffffL) return fail(QGEMM_EUNSUPPORTED, "too many tiles");
    hipLaunchKernelGGL((qg::moe_kernel<FMT, BM, BN, WM, WN, XS, SWI, CMB>), dim3((unsigned)grid), dim3(WM * WN * 64), 0,
                       s, a, ep);
    const int rc = check_launch("qgemm_moe");
    if (rc != QGEMM_OK) return rc;
  }
  return QGEMM_OK;
}

// Column tile width of the configuration launch_moe picks (the fused combine counts arrivals per
// (token, column tile)).
inline int moe_tile_bn(long M, int E) { return (M / E) <= 32 ? 128 : 256; }

// Tile from the mean rows per expert (the host does not see the routing): groups of about
// 100-200 rows fit one 192-row tile each; larger groups use 256-row tiles. Short prompts (at
// most 32 rows per expert on average) use four-wave tiles with 128 columns: twice the
// workgroups of the 256-wide tiles over the few active experts' weights, so the CUs fill
// (measured at T=128, E=128, top-8: gate/up + SiLU 66.5 against 73 us, down 31 against 34 us;
// at T=2048 the same tile is slower, 196 against 159 us and 125 against 108 us). The fused
// gate/up tile is 64 rows high there (three workgroups per CU, so the whole launch runs in one
// round: 52-53 against 67-68 us); the plain tile stays 128 rows high (down 31-33 against 33-34 us
// with 64 rows).
template <int FMT, bool SWI = false, bool CMB = false>
int launch_moe(qg::TileArgs a, const void* const* wq, const void* const* sc, int E, hipStream_t s) {
  const long mean_rows = (long)a.M / E;
  if (mean_rows <= 32) return launch_moe_cfg<FMT, SWI ? 64 : 128, 128, 2, 2, 2, SWI, CMB>(a, wq, sc, E, s);
  if (mean_rows > 192) return launch_moe_cfg<FMT, 256, 256, 2, 4, 2, SWI, CMB>(a, wq, sc, E, s);
  return launch_moe_cfg<FMT, 192, 256, 2, 4, 2, SWI, CMB>(a, wq, sc, E, s);
}

// ---------------------------------------------------------------------------
// MoE workspace (per device): bucketing output, per-block counts, error flag
// ---------------------------------------------------------------------------

struct Workspace {
  int32_t* perm = nullptr;
  size_t perm_cap = 0;
  int32_t* counts = nullptr;
  size_t counts_cap = 0;
  int32_t* flag = nullptr;
  int seq = 0;
  int32_t* arrivals = nullptr;   // fused combine: per (token, column tile) arrival counters
  size_t arrivals_cap = 0;
};

std::mutex g_ws_mutex;
std::vector<Workspace> g_ws;

int grow(int32_t** p, size_t* cap, size_t need) {
  if (*cap >= need) return QGEMM_OK;
  if (*p != nullptr) {
    (void)hipFree(*p);   // hipFree waits for outstanding work that may still read the buffer
    *p = nullptr;
    *cap = 0;
  }
  size_t want = need < 4096 ? 4096 : need;
  if (hipMalloc(reinterpret_cast<void**>(p), want * sizeof(int32_t)) != hipSuccess) {
    (void)hipGetLastError();
    return fail(QGEMM_EHIP, "hipMalloc of %zu bytes for the MoE workspace failed", want * sizeof(int32_t));
  }
  *cap = want;
  return QGEMM_OK;
}

int bucket_geometry(int n, int* chunk, int* nblk) {
  int c = 512;   // one or two rounds of the scatter per block, and >= 100 blocks at 64K slots
  long nb = ((long)n + c - 1) / c;
  if (nb > 1024) {
    c = (int)((((long)n + 1023) / 1024 + 255) / 256 * 256);
    nb = ((long)n + c - 1) / c;
  }
  *chunk = c;
  *nblk = (int)nb;
  return QGEMM_OK;
}

constexpr int kMaxE = 4096;

int enqueue_bucket(const int32_t* idx, const int32_t* offsets, int32_t* perm, int n, int E, int32_t* counts,
                   int32_t* flag, int seq, float* ypoison, int N, hipStream_t s) {
  int chunk, nblk;
  bucket_geometry(n, &chunk, &nblk);
  const size_t lds = (size_t)E * sizeof(int32_t);
  hipLaunchKernelGGL(qg::bucket_count_kernel, dim3(nblk), dim3(qg::kBucketThreads), lds, s, idx, n, E, chunk, counts);
  int rc = check_launch("moe bucket count");
  if (rc != QGEMM_OK) return rc;
  hipLaunchKernelGGL(qg::bucket_scatter_kernel, dim3(nblk), dim3(qg::kBucketThreads), lds, s, idx, offsets, n, E,
                     chunk, counts, nblk, perm, flag, seq, ypoison, N);
  return check_launch("moe bucket scatter");
}

Workspace* workspace_for_current_device(int* dev_out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  if ((int)g_ws.size() <= dev) g_ws.resize(dev + 1);
  *dev_out = dev;
  return &g_ws[dev];
}

int moe_args_check(const void* x, const void* idx_or_perm, const int32_t* offsets, const void* const* wq,
                   const void* const* scales, const float* y, int T, int E, int topk, int N, int K, int fmt) {
  int rc = check_common(N, K, fmt);
  if (rc != QGEMM_OK) return rc;
  if (T < 0) return fail(QGEMM_EINVAL, "T must be >= 0 (got %d)", T);
  if (E < 1) return fail(QGEMM_EINVAL, "E must be >= 1 (got %d)", E);
  if (E > kMaxE) return fail(QGEMM_EUNSUPPORTED, "E = %d exceeds the supported %d experts", E, kMaxE);
  if (topk < 1 || topk > E) return fail(QGEMM_EINVAL, "topk must lie in [1, E] (got %d)", topk);
  if ((long)T * topk > 0x7fffffffL) return fail(QGEMM_EUNSUPPORTED, "T*topk too large");
  if ((long)T * topk * N > 0x7fffffffffffL || (long)T * K > 0x7fffffffL || ((long)T + 1) * K * 2 + 256 >= 0xFFFFFFF0L)
    return fail(QGEMM_EUNSUPPORTED, "problem too large");
  if (T == 0) return QGEMM_OK;
  if (!x || !idx_or_perm || !offsets || !wq || !scales || !y) return fail(QGEMM_EINVAL, "null pointer argument");
  if (!aligned16(x) || !aligned16(y) || !aligned16(idx_or_perm) || !aligned16(offsets))
    return fail(QGEMM_EALIGN, "x, y and routing tables must be 16-byte aligned");
  for (int e = 0; e < E; ++e) {
    if (!wq[e] || !scales[e]) return fail(QGEMM_EINVAL, "null weight or scale pointer for expert %d", e);
    if (!aligned16(wq[e])) return fail(QGEMM_EALIGN, "weights of expert %d are not 16-byte aligned", e);
    if ((reinterpret_cast<uintptr_t>(scales[e]) & 1u) != 0)
      return fail(QGEMM_EALIGN, "scales of expert %d are not 2-byte aligned", e);
  }
  return QGEMM_OK;
}

// ---------------------------------------------------------------------------
// allocation-free MoE entry point: the bucketing buffers live in a static device array
// ---------------------------------------------------------------------------

constexpr int kNoAllocMaxSlots = 1 << 18;    // token slots (T * topk): the permutation
constexpr int kNoAllocMaxCounts = 1 << 18;   // per-block expert histograms (blocks x E)
constexpr int kNoAllocFlag = kNoAllocMaxSlots + kNoAllocMaxCounts;   // error flag (sequence number)
constexpr int kMaxDevices = 64;

std::mutex g_scratch_mutex;
int32_t* g_scratch_dev[kMaxDevices] = {};    // device address of `scratch` on each device
int g_scratch_seq[kMaxDevices] = {};

bool validate_env() {
  const char* v = getenv("QGEMM_VALIDATE");
  return v != nullptr && v[0] == '1';
}

}  // namespace

extern "C" {

int qgemm_version(void) { return (1 << 16) | 0; }

const char* qgemm_last_error(void) { return g_last_error.c_str(); }

int qgemm_dense(const void* x, const void* wq, const void* scales, float* y, int M, int N, int K, int fmt,
                hipStream_t stream) {
  int rc = check_common(N, K, fmt);
  if (rc != QGEMM_OK) return rc;
  if (M < 0) return fail(QGEMM_EINVAL, "M must be >= 0 (got %d)", M);
  if ((long)M * K > 0x7fffffffL || (long)N * K > 0x7fffffffL || (long)M * N > 0x7fffffffL)
    return fail(QGEMM_EUNSUPPORTED, "an operand has 2^31 or more elements");
  if (M == 0) return ok();
  if (!x || !wq || !scales || !y) return fail(QGEMM_EINVAL, "null pointer argument");
  if (!aligned16(x) || !aligned16(wq) || !aligned16(y))
    return fail(QGEMM_EALIGN, "x, wq and y must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(scales) & 1u) != 0) return fail(QGEMM_EALIGN, "scales must be 2-byte aligned");
  (void)hipGetLastError();
  qg::TileArgs a{};
  a.x = static_cast<const uint16_t*>(x);
  a.y = y;
  a.M = M;
  a.N = N;
  a.K = K;
  rc = (fmt == QGEMM_Q8) ? dense_dispatch<qg::kQ8>(a, wq, scales, stream)
                         : dense_dispatch<qg::kQ4>(a, wq, scales, stream);
  return rc == QGEMM_OK ? ok() : rc;
}

int qgemm_moe_bucket(const int32_t* token_expert_idx, const int32_t* expert_offsets, int32_t* perm, int n_assign,
                     int E, hipStream_t stream) {
  if (n_assign < 0) return fail(QGEMM_EINVAL, "n_assign must be >= 0");
  if (E < 1) return fail(QGEMM_EINVAL, "E must be >= 1");
  if (E > kMaxE) return fail(QGEMM_EUNSUPPORTED, "E = %d exceeds the supported %d experts", E, kMaxE);
  if (n_assign == 0) return ok();
  if (!token_expert_idx || !expert_offsets || !perm) return fail(QGEMM_EINVAL, "null pointer argument");
  if (!aligned16(token_expert_idx) || !aligned16(expert_offsets) || !aligned16(perm))
    return fail(QGEMM_EALIGN, "routing tables must be 16-byte aligned");
  std::lock_guard<std::mutex> lock(g_ws_mutex);
  int dev;
  Workspace* ws = workspace_for_current_device(&dev);
  if (!ws) return fail(QGEMM_EHIP, "hipGetDevice failed");
  int chunk, nblk;
  bucket_geometry(n_assign, &chunk, &nblk);
  int rc = grow(&ws->counts, &ws->counts_cap, (size_t)nblk * E);
  if (rc != QGEMM_OK) return rc;
  size_t one = 0;
  if (ws->flag == nullptr) {
    rc = grow(&ws->flag, &one, 1);
    if (rc != QGEMM_OK) return rc;
  }
  (void)hipGetLastError();
  rc = enqueue_bucket(token_expert_idx, expert_offsets, perm, n_assign, E, ws->counts, ws->flag, 0, nullptr, 0,
                      stream);
  return rc == QGEMM_OK ? ok() : rc;
}

int qgemm_moe_grouped(const void* x, const int32_t* perm, const int32_t* expert_offsets, const void* const* wq,
                      const void* const* scales, float* y, int T, int E, int topk, int N, int K, int fmt,
                      hipStream_t stream) {
  int rc = moe_args_check(x, perm, expert_offsets, wq, scales, y, T, E, topk, N, K, fmt);
  if (rc != QGEMM_OK || T == 0) return rc == QGEMM_OK ? ok() : rc;
  (void)hipGetLastError();
  qg::TileArgs a{};
  a.x = static_cast<const uint16_t*>(x);
  a.y = y;
  a.M = T * topk;
  a.N = N;
  a.K = K;
  a.perm = perm;
  a.offsets = expert_offsets;
  a.topk = topk;
  a.T = T;
  rc = (fmt == QGEMM_Q8) ? launch_moe<qg::kQ8>(a, wq, scales, E, stream)
                         : launch_moe<qg::kQ4>(a, wq, scales, E, stream);
  return rc == QGEMM_OK ? ok() : rc;
}

int qgemm_moe_gate_up_swiglu(const void* x, const int32_t* perm, const int32_t* expert_offsets,
                              const void* const* wq, const void* const* scales, void* h, int T, int E, int topk,
                              int inter, int K, int fmt, hipStream_t stream) {
  if (inter < 1 || inter > 0x3fffffff) return fail(QGEMM_EINVAL, "inter must be >= 1 (got %d)", inter);
  if ((long)T * topk * inter > 0x7fffffffffffL) return fail(QGEMM_EUNSUPPORTED, "problem too large");
  // the y pointer check of the shared validation stands for h
  int rc = moe_args_check(x, perm, expert_offsets, wq, scales, static_cast<const float*>(h), T, E, topk, 2 * inter, K,
                          fmt);
  if (rc != QGEMM_OK || T == 0) return rc == QGEMM_OK ? ok() : rc;
  if ((long)2 * inter * (K / 32) * 2 > 0xffffffffL || (long)2 * inter * K > 0xffffffffL)
    return fail(QGEMM_EUNSUPPORTED, "an expert's weights span 4 GiB or more");
  (void)hipGetLastError();
  qg::TileArgs a{};
  a.x = static_cast<const uint16_t*>(x);
  a.y = nullptr;
  a.M = T * topk;
  a.N = 2 * inter;
  a.K = K;
  a.perm = perm;
  a.offsets = expert_offsets;
  a.topk = topk;
  a.T = T;
  a.swi_inter = inter;
  a.h = static_cast<uint16_t*>(h);
  rc = (fmt == QGEMM_Q8) ? launch_moe<qg::kQ8, true>(a, wq, scales, E, stream)
                         : launch_moe<qg::kQ4, true>(a, wq, scales, E, stream);
  return rc == QGEMM_OK ? ok() : rc;
}

int qgemm_moe(const void* x, const int32_t* token_expert_idx, const int32_t* expert_offsets, const void* const* wq,
              const void* const* scales, float* y, int T, int E, int topk, int N, int K, int fmt,
              hipStream_t stream) {
  int rc = moe_args_check(x, token_expert_idx, expert_offsets, wq, scales, y, T, E, topk, N, K, fmt);
  if (rc != QGEMM_OK || T == 0) return rc == QGEMM_OK ? ok() : rc;
  const int n = T * topk;
  int seq;
  int32_t* perm;
  int32_t* flag;
  {
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    int dev;
    Workspace* ws = workspace_for_current_device(&dev);
    if (!ws) return fail(QGEMM_EHIP, "hipGetDevice failed");
    int chunk, nblk;
    bucket_geometry(n, &chunk, &nblk);
    rc = grow(&ws->perm, &ws->perm_cap, (size_t)n);
    if (rc == QGEMM_OK) rc = grow(&ws->counts, &ws->counts_cap, (size_t)nblk * E);
    if (rc == QGEMM_OK && ws->flag == nullptr) {
      size_t one = 0;
      rc = grow(&ws->flag, &one, 1);
      if (rc == QGEMM_OK) {
        if (hipMemset(ws->flag, 0, sizeof(int32_t)) != hipSuccess) rc = fail(QGEMM_EHIP, "hipMemset failed");
      }
    }
    if (rc != QGEMM_OK) return rc;
    ws->seq = ws->seq == 0x7fffffff ? 1 : ws->seq + 1;
    seq = ws->seq;
    perm = ws->perm;
    flag = ws->flag;
    (void)hipGetLastError();
    rc = enqueue_bucket(token_expert_idx, expert_offsets, perm, n, E, ws->counts, flag, seq, y, N, stream);
    if (rc != QGEMM_OK) return rc;
  }
  qg::TileArgs a{};
  a.x = static_cast<const uint16_t*>(x);
  a.y = y;
  a.M = n;
  a.N = N;
  a.K = K;
  a.perm = perm;
  a.offsets = expert_offsets;
  a.topk = topk;
  a.T = T;
  rc = (fmt == QGEMM_Q8) ? launch_moe<qg::kQ8>(a, wq, scales, E, stream)
                         : launch_moe<qg::kQ4>(a, wq, scales, E, stream);
  if (rc != QGEMM_OK) return rc;
  if (validate_env()) {
    if (hipStreamSynchronize(stream) != hipSuccess) return fail(QGEMM_EHIP, "hipStreamSynchronize failed");
    int32_t h = 0;
    if (hipMemcpy(&h, flag, sizeof h, hipMemcpyDeviceToHost) != hipSuccess) return fail(QGEMM_EHIP, "hipMemcpy failed");
    if (h == seq) return fail(QGEMM_EINVAL, "token_expert_idx and expert_offsets disagree");
  }
  return ok();
}

int qgemm_moe_down_combine(const void* h, const int32_t* perm, const int32_t* expert_offsets, const void* const* wq,
                           const void* const* scales, const float* route_w, float* y2, float* out, int T, int E,
                           int topk, int N, int K, int fmt, hipStream_t stream) {
  if (T < 0 || topk < 1) return fail(QGEMM_EINVAL, "T must be >= 0 and topk >= 1");
  if ((long)T * topk > 0x7fffffffL) return fail(QGEMM_EUNSUPPORTED, "T*topk too large");
  const int A = T * topk;
  // the down projection proper: A rows of h, identity gather
  int rc = moe_args_check(h, perm, expert_offsets, wq, scales, y2, A, E, 1, N, K, fmt);
  if (rc != QGEMM_OK) return rc;
  if (topk > E) return fail(QGEMM_EINVAL, "topk must lie in [1, E] (got %d)", topk);
  if (N % 4 != 0) return fail(QGEMM_EINVAL, "N must be a multiple of 4 (got %d)", N);
  if ((double)A * N * 4.0 >= 4294967296.0) return fail(QGEMM_EUNSUPPORTED, "y2 must span less than 4 GiB");
  if (T == 0) return ok();
  if (!route_w || !out) return fail(QGEMM_EINVAL, "null pointer argument");
  if (!aligned16(route_w) || !aligned16(out)) return fail(QGEMM_EALIGN, "route_w and out must be 16-byte aligned");
  const int bn = moe_tile_bn(A, E);
  const long nctr = (long)T * ((N + bn - 1) / bn);
  int32_t* ctr = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    int dev;
    Workspace* ws = workspace_for_current_device(&dev);
    if (!ws) return fail(QGEMM_EHIP, "hipGetDevice failed");
    rc = grow(&ws->arrivals, &ws->arrivals_cap, (size_t)nctr);
    if (rc != QGEMM_OK) return rc;
    ctr = ws->arrivals;
  }
  (void)hipGetLastError();
  // counters start at zero every call (a fill kernel, not a memset node, so the call can be captured)
  hipLaunchKernelGGL(qg::fill_i32_kernel, dim3((unsigned)((nctr + 1023) / 1024)), dim3(256), 0, stream, ctr, nctr, 0);
  rc = check_launch("qgemm_moe_down_combine (arrival counters)");
  if (rc != QGEMM_OK) return rc;
  qg::TileArgs a{};
  a.x = static_cast<const uint16_t*>(h);
  a.y = y2;
  a.M = A;
  a.N = N;
  a.K = K;
  a.perm = perm;
  a.offsets = expert_offsets;
  a.topk = 1;
  a.T = A;
  a.cmb_topk = topk;
  a.route_w = route_w;
  a.out = out;
  a.counters = ctr;
  rc = (fmt == QGEMM_Q8) ? launch_moe<qg::kQ8, false, true>(a, wq, scales, E, stream)
                         : launch_moe<qg::kQ4, false, true>(a, wq, scales, E, stream);
  return rc == QGEMM_OK ? ok() : rc;
}

int qgemm_moe_noalloc(const void* x, const int32_t* token_expert_idx, const int32_t* expert_offsets,
                      const void* const* wq, const void* const* scales, float* y, int T, int E, int topk, int N,
                      int K, int fmt, hipStream_t stream) {
  int rc = moe_args_check(x, token_expert_idx, expert_offsets, wq, scales, y, T, E, topk, N, K, fmt);
  if (rc != QGEMM_OK || T == 0) return rc == QGEMM_OK ? ok() : rc;
  const int n = T * topk;
  int chunk, nblk;
  bucket_geometry(n, &chunk, &nblk);
  if (n > kNoAllocMaxSlots)
    return fail(QGEMM_EUNSUPPORTED, "qgemm_moe_noalloc: T*topk = %d exceeds the static scratch (%d token slots)", n,
                kNoAllocMaxSlots);
  if ((long)nblk * E > kNoAllocMaxCounts)
    return fail(QGEMM_EUNSUPPORTED,
                "qgemm_moe_noalloc: %d bucketing blocks x %d experts exceed the static scratch (%d counts)", nblk, E,
                kNoAllocMaxCounts);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return fail(QGEMM_EHIP, "hipGetDevice failed");
  }
  if (dev < 0 || dev >= kMaxDevices) return fail(QGEMM_EUNSUPPORTED, "device %d beyond the supported %d", dev, kMaxDevices);
  int32_t* base;
  int seq;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_dev[dev] == nullptr) {
      // once per device, with that device current: the address of this device's copy of the array
      void* p = nullptr;
      const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || p == nullptr) {
        (void)hipGetLastError();
        return fail(QGEMM_EHIP, "hipGetSymbolAddress of the static scratch failed: %s", hipGetErrorString(e));
      }
      g_scratch_dev[dev] = static_cast<int32_t*>(p);
    }
    base = g_scratch_dev[dev];
    g_scratch_seq[dev] = g_scratch_seq[dev] == 0x7fffffff ? 1 : g_scratch_seq[dev] + 1;
    seq = g_scratch_seq[dev];
  }
  int32_t* perm = base;
  int32_t* counts = base + kNoAllocMaxSlots;
  int32_t* flag = base + kNoAllocFlag;
  (void)hipGetLastError();
  // every entry of perm and of the histograms is written by the bucketing kernels before it is
  // read; the flag is compared with this call's sequence number, so nothing needs clearing
  rc = enqueue_bucket(token_expert_idx, expert_offsets, perm, n, E, counts, flag, seq, y, N, stream);
  if (rc != QGEMM_OK) return rc;
  qg::TileArgs a{};
  a.x = static_cast<const uint16_t*>(x);
  a.y = y;
  a.M = n;
  a.N = N;
  a.K = K;
  a.perm = perm;
  a.offsets = expert_offsets;
  a.topk = topk;
  a.T = T;
  rc = (fmt == QGEMM_Q8) ? launch_moe<qg::kQ8>(a, wq, scales, E, stream) : launch_moe<qg::kQ4>(a, wq, scales, E, stream);
  return rc == QGEMM_OK ? ok() : rc;
}

int qgemm_swiglu(const float* y1, void* h, int rows, int inter, hipStream_t stream) {
  if (rows < 0 || inter < 8 || inter % 8 != 0)
    return fail(QGEMM_EINVAL, "rows must be >= 0 and inter a positive multiple of 8");
  if (rows == 0) return ok();
  if (!y1 || !h) return fail(QGEMM_EINVAL, "null pointer argument");
  if (!aligned16(y1) || !aligned16(h)) return fail(QGEMM_EALIGN, "y1 and h must be 16-byte aligned");
  const long groups = (long)rows * (inter / 8);
  const long blocks = (groups + 255) / 256;
  if (blocks > 0x7fffffffL) return fail(QGEMM_EUNSUPPORTED, "problem too large");
  (void)hipGetLastError();
  hipLaunchKernelGGL(qg::swiglu_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, y1,
                     static_cast<uint16_t*>(h), groups, inter);
  const int rc = check_launch("qgemm_swiglu");
  return rc == QGEMM_OK ? ok() : rc;
}

int qgemm_moe_combine(const float* y2, const float* route_w, float* out, int T, int topk, int N, hipStream_t stream) {
  if (T < 0 || topk < 1 || N < 4 || N % 4 != 0)
    return fail(QGEMM_EINVAL, "T must be >= 0, topk >= 1 and N a positive multiple of 4");
  if (T == 0) return ok();
  if (!y2 || !route_w || !out) return fail(QGEMM_EINVAL, "null pointer argument");
  if (!aligned16(y2) || !aligned16(out) || !aligned16(route_w))
    return fail(QGEMM_EALIGN, "y2, route_w and out must be 16-byte aligned");
  const int v = (N % 8 == 0) ? 8 : 4;
  const long groups = (long)T * (N / v);
  const long blocks = (groups + 255) / 256;
  if (blocks > 0x7fffffffL) return fail(QGEMM_EUNSUPPORTED, "problem too large");
  (void)hipGetLastError();
  // column mapping by where y2 will come from: a y2 that fits well inside the 256 MB last-level
  // cache (just written by the down projection) reads faster with wave-contiguous 16-byte
  // accesses, a larger one (streamed from HBM) with each thread's outputs consecutive (measured:
  // 128 MiB y2 22 us against 29 us, 512 MiB 110 us against 114 us)
  const bool spread = (double)T * topk * N * 4.0 <= 192.0 * 1024 * 1024;
  // top-8 routing (the paper's MoE models) gets a kernel with every slot's loads issued up front
  auto launch = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(256), 0, stream, y2, route_w, out, groups, topk, N);
  };
  if (v == 8 && topk == 8)
    spread ? launch(qg::combine_kernel<8, 8, true>) : launch(qg::combine_kernel<8, 8, false>);
  else if (v == 8)
    spread ? launch(qg::combine_kernel<8, 0, true>) : launch(qg::combine_kernel<8, 0, false>);
  else
    spread ? launch(qg::combine_kernel<4, 0, true>) : launch(qg::combine_kernel<4, 0, false>);
  const int rc = check_launch("qgemm_moe_combine");
  return rc == QGEMM_OK ? ok() : rc;
}

int qgemm_attention_prefill(const void* q, const void* k, const void* v, void* o, int B, int S, int H, int Hkv, int D,
                            float scale, int causal, hipStream_t stream) {
  if (B < 0 || S < 0) return fail(QGEMM_EINVAL, "B and S must be >= 0 (got %d, %d)", B, S);
  if (H < 1 || Hkv < 1 || H % Hkv != 0)
    return fail(QGEMM_EINVAL, "H and Hkv must be >= 1 with H a multiple of Hkv (got %d, %d)", H, Hkv);
  if (D != 64 && D != 128) return fail(QGEMM_EUNSUPPORTED, "head dimension must be 64 or 128 (got %d)", D);
  if (causal != 0 && causal != 1) return fail(QGEMM_EINVAL, "causal must be 0 or 1 (got %d)", causal);
  if (!(scale > 0.0f) || !std::isfinite(scale)) return fail(QGEMM_EINVAL, "scale must be finite and > 0");
  if ((long)S * H * D > 0x7fffffffL) return fail(QGEMM_EUNSUPPORTED, "S*H*D must be below 2^31");
  const long nqb = (S + qg::kAttnBQ - 1) / qg::kAttnBQ;
  if ((long)B * H * nqb > 0x7fffffffL) return fail(QGEMM_EUNSUPPORTED, "too many workgroups");
  if (B == 0 || S == 0) return ok();
  if (!q || !k || !v || !o) return fail(QGEMM_EINVAL, "null pointer argument");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return fail(QGEMM_EALIGN, "q, k, v and o must be 16-byte aligned");
  (void)hipGetLastError();
  qg::AttnArgs a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.o = static_cast<uint16_t*>(o);
  a.B = B;
  a.S = S;
  a.H = H;
  a.Hkv = Hkv;
  a.sl2 = (float)((double)scale * 1.4426950408889634);   // exp(x) = exp2(x log2 e)
  const dim3 grid((unsigned)(B * H * nqb)), block(qg::kAttnThreads);
  if (D == 128) {
    if (causal) hipLaunchKernelGGL((qg::attn_fwd_kernel<128, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((qg::attn_fwd_kernel<128, false>), grid, block, 0, stream, a);
  } else {
    if (causal) hipLaunchKernelGGL((qg::attn_fwd_kernel<64, true>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((qg::attn_fwd_kernel<64, false>), grid, block, 0, stream, a);
  }
  const int rc = check_launch("qgemm_attention_prefill");
  return rc == QGEMM_OK ? ok() : rc;
}

int qgemm_probe_mfma_clock(int iters, double* sclk_mhz, double* mfma_tflops, hipStream_t stream) {
  if (iters < 1 || !sclk_mhz || !mfma_tflops) return fail(QGEMM_EINVAL, "iters must be >= 1 and outputs non-null");
  int dev = 0, ncu = 0, rt_khz = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipDeviceGetAttribute(&rt_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess || ncu < 1 || rt_khz < 1) {
    (void)hipGetLastError();
    return fail(QGEMM_EHIP, "device attribute query failed");
  }
  long long* stamps = nullptr;
  float* sink = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = QGEMM_OK;
  if (hipMalloc(reinterpret_cast<void**>(&stamps), (size_t)ncu * 4 * sizeof(long long)) != hipSuccess ||
      hipMalloc(reinterpret_cast<void**>(&sink), qg::kProbeThreads * sizeof(float)) != hipSuccess ||
      hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
    rc = fail(QGEMM_EHIP, "probe set-up failed");
  }
  std::vector<long long> h((size_t)ncu * 4);
  float ms = 0.0f;
  if (rc == QGEMM_OK) {
    (void)hipGetLastError();
    (void)hipEventRecord(e0, stream);
    hipLaunchKernelGGL(qg::mfma_clock_probe_kernel, dim3(ncu), dim3(qg::kProbeThreads), 0, stream, stamps, iters, sink);
    rc = check_launch("qgemm_probe_mfma_clock");
    (void)hipEventRecord(e1, stream);
    if (rc == QGEMM_OK) {
      if (hipStreamSynchronize(stream) != hipSuccess || hipEventElapsedTime(&ms, e0, e1) != hipSuccess ||
          hipMemcpy(h.data(), stamps, h.size() * sizeof(long long), hipMemcpyDeviceToHost) != hipSuccess)
        rc = fail(QGEMM_EHIP, "probe read-back failed");
    }
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (stamps) (void)hipFree(stamps);
  if (sink) (void)hipFree(sink);
  (void)hipGetLastError();
  if (rc != QGEMM_OK) return rc;
  std::vector<double> mhz;
  for (int b = 0; b < ncu; ++b) {
    const double dc = (double)(h[4 * b + 1] - h[4 * b]);
    const double dt = (double)(h[4 * b + 3] - h[4 * b + 2]) / ((double)rt_khz * 1e3);   // seconds
    if (dt > 0 && dc > 0) mhz.push_back(dc / dt * 1e-6);
  }
  if (mhz.empty() || !(ms > 0.0f)) return fail(QGEMM_EHIP, "probe produced no timing");
  std::sort(mhz.begin(), mhz.end());
  *sclk_mhz = mhz[mhz.size() / 2];
  const double flop = (double)ncu * (qg::kProbeThreads / 64) * (double)iters * 4.0 * 32.0 * 32.0 * 16.0 * 2.0;
  *mfma_tflops = flop / ((double)ms * 1e-3) / 1e12;
  return ok();
}

int qgemm_release(void) {
  std::lock_guard<std::mutex> lock(g_ws_mutex);
  int cur = 0;
  (void)hipGetDevice(&cur);
  for (size_t d = 0; d < g_ws.size(); ++d) {
    Workspace& w = g_ws[d];
    if (!w.perm && !w.counts && !w.flag && !w.arrivals) continue;
    (void)hipSetDevice((int)d);
    if (w.perm) (void)hipFree(w.perm);
    if (w.counts) (void)hipFree(w.counts);
    if (w.flag) (void)hipFree(w.flag);
    if (w.arrivals) (void)hipFree(w.arrivals);
    w = Workspace{};
  }
  {
    std::lock_guard<std::mutex> split_lock(g_split_mutex);
    for (size_t d = 0; d < g_split_ws.size(); ++d) {
      if (!g_split_ws[d].first) continue;
      (void)hipSetDevice((int)d);
      (void)hipFree(g_split_ws[d].first);
      g_split_ws[d] = {nullptr, 0};
    }
  }
  (void)hipSetDevice(cur);
  (void)hipGetLastError();
  return ok();
}

}  // extern "C"
