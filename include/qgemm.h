/*
 * qgemm.h - C ABI of the MI355X (gfx950) block-quantised prefill GEMM library.
 *
 * The library computes the prompt-processing (prefill) matrix multiplies the
 * paper routes onto matrix units (Section 3.1): dense projection GEMMs over
 * 4-bit / 8-bit block-quantised weights, and the MoE expert GEMM that
 * evaluates each active expert's projection over the tokens routed to it,
 * plus the SiLU-gated activation between the MoE projections (Section 3.1,
 * fused gate/up item) and the router-weighted combine of the experts' outputs.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers are DEVICE pointers (memory the HIP runtime of this process
 *   allocated on the current device) unless the comment says HOST.
 * - Arrays are dense and row-major; no strides. Every device pointer must be
 *   16-byte aligned, except fp16 scale arrays, which need 2-byte alignment
 *   (QGEMM_EALIGN otherwise).
 * - Work is enqueued on `stream` (0 = the null stream) and the call returns
 *   without synchronising; device faults surface at the caller's next sync.
 *   The caller keeps every buffer alive until the stream has passed the call.
 * - Outputs are written, never accumulated into, and must not alias inputs.
 * - Return value: QGEMM_OK (0) or a negative QGEMM_E* code. On an error return
 *   nothing has been enqueued and no output is written;
 *   qgemm_last_error() gives a message. No entry point throws.
 * - A zero-sized problem (M, T or rows == 0) returns QGEMM_OK and launches
 *   nothing.
 *
 * Storage formats (the paper names 4-bit and 8-bit block quantisation without a
 * byte layout; this is the layout the library reads):
 * - activations x: bf16 [rows][K].
 * - QGEMM_Q8 weights: int8 [N][K]; element (n, k) means q * s.
 * - QGEMM_Q4 weights: uint8 [N][K/2]; byte j of a row holds element 2j in
 *   bits 0-3 and element 2j+1 in bits 4-7; a nibble u means (u - 8) * s.
 * - scales: fp16 [N][K/32]; s = scales[n][k / 32] (one scale per 32
 *   consecutive K elements of a row).
 * - K must be a multiple of 32.
 * - results: fp32, y[m][n] = sum_k x[m][k] * s[n][k/32] * q[n][k]; the
 *   library rounds each dequantised weight to bf16 and accumulates in fp32.
 */
#ifndef QGEMM_H
#define QGEMM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#ifndef __HIP_INCLUDE_HIP_HIP_RUNTIME_API_H__
typedef struct ihipStream_t* hipStream_t;
#endif

enum qgemm_fmt { QGEMM_Q8 = 0, QGEMM_Q4 = 1 };

enum qgemm_status {
  QGEMM_OK = 0,
  QGEMM_EINVAL = -1,       /* bad size, format, null pointer or routing table */
  QGEMM_EALIGN = -2,       /* a device pointer is not 16-byte aligned */
  QGEMM_EUNSUPPORTED = -3, /* a size beyond what the library handles */
  QGEMM_EHIP = -4          /* the HIP runtime reported an error */
};

/*
 * Dense block-quantised GEMM (Section 3.1, dense GEMM item):
 *   y[M][N] = x[M][K] . dequant(wq, scales)^T
 * x: bf16 [M][K]; wq: int8 [N][K] (Q8) or uint8 [N][K/2] (Q4);
 * scales: fp16 [N][K/32]; y: fp32 [M][N].
 * Sizes: M >= 0, 1 <= N, 32 <= K, K % 32 == 0, every element count < 2^31.
 * When few output tiles meet a long K, the call splits K over several
 * workgroups and sums their fp32 partials in split order (deterministic) in a
 * library-owned workspace (grown on first use, freed by qgemm_release);
 * concurrent calls on different streams must not share it.
 * M <= 16 (decode and speculative-draft verification, the memory-bound
 * regime of Section 2.3 and the batched verification of Section 5.2) takes a
 * separate bandwidth-oriented kernel: weights dequantised straight into
 * matrix-core registers, K split over waves (and over workgroups when N is
 * small, through the same workspace). The same kernel, in blocks of 16
 * activation rows, serves 16 < M <= 128 when ceil(N/128) times the number of
 * 16-row blocks (rounded up to 2, 4 or 8) is at most 512: short prompts whose
 * few 128x128 output tiles would leave most CUs idle. Its results are bitwise
 * reproducible but not bitwise equal to the tile kernels' (another summation
 * order).
 */
int qgemm_dense(const void* x, const void* wq, const void* scales, float* y,
                int M, int N, int K, int fmt, hipStream_t stream);

/*
 * MoE expert GEMM (Section 3.1, MoE expert GEMM item): every token slot
 * ("assignment") a = t*topk + j is multiplied by the weights of its expert:
 *   y[a][:] = dequant(wq[e], scales[e]) . x[a / topk][:],  e = token_expert_idx[a]
 * Only experts with at least one assignment read their weights.
 * x: bf16 [T][K].
 * token_expert_idx: int32 [T*topk], values in [0, E).
 * expert_offsets: int32 [E+1], exclusive prefix sum of the per-expert
 *   assignment counts (offsets[0] == 0, offsets[E] == T*topk).
 * wq, scales: HOST arrays of E device pointers, each laid out as for
 *   qgemm_dense with the same N and K.
 * y: fp32 [T*topk][N], in assignment (token-slot) order.
 * Sizes: 1 <= E <= 4096, 1 <= topk <= E, T*topk < 2^31, T*K < 2^31.
 * The call buckets the assignments by expert into a library-owned workspace
 * (grown on first use, then reused; freed by qgemm_release) and runs the
 * grouped GEMM. Routing tables that disagree with each other are a caller
 * error: every access stays in bounds, and the rows of y that depend on the
 * inconsistent expert are written as NaN. With the environment variable
 * QGEMM_VALIDATE=1 the call synchronises `stream` and returns QGEMM_EINVAL
 * in that case.
 * Calls that share the workspace are ordered only by their streams: do not
 * run two qgemm_moe calls concurrently on different streams.
 */
int qgemm_moe(const void* x, const int32_t* token_expert_idx,
              const int32_t* expert_offsets, const void* const* wq,
              const void* const* scales, float* y, int T, int E, int topk,
              int N, int K, int fmt, hipStream_t stream);

/*
 * qgemm_moe for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same arguments, results bitwise equal to qgemm_moe, and no hipMalloc, hipFree
 * or other allocation on any call. The bucketing buffers (permutation,
 * per-block expert histograms, error flag) live in a static device array of
 * 2 MiB + 256 bytes that each device holds until the process ends; the first
 * call on a device looks up its address there. Limits: T*topk <= 262144 and
 * ceil-blocks(T*topk) * E <= 262144 (the bucketing uses blocks of 512 slots,
 * at most 1024 blocks); larger problems return QGEMM_EUNSUPPORTED before
 * anything is enqueued. Every call on a device shares that device's array and
 * leaves its contents behind: calls that can overlap on one device (other
 * streams, other host threads) race and must be ordered by the caller.
 * QGEMM_VALIDATE is not consulted (the call never synchronises); inconsistent
 * routing tables still give NaN rows as for qgemm_moe.
 */
int qgemm_moe_noalloc(const void* x, const int32_t* token_expert_idx,
                      const int32_t* expert_offsets, const void* const* wq,
                      const void* const* scales, float* y, int T, int E, int topk,
                      int N, int K, int fmt, hipStream_t stream);

/*
 * The two halves of qgemm_moe, for callers that keep their own bucketing
 * buffer (the MoE expert GEMM of Section 3.1 needs each expert's routed
 * token list).
 * qgemm_moe_bucket: perm: int32 [n_assign], caller-owned. Writes the
 *   assignments grouped by expert: perm[expert_offsets[e] + r] is the r-th
 *   assignment (in increasing order) routed to expert e. Stable and
 *   deterministic. Entries for an expert whose count disagrees with
 *   expert_offsets are written as -1.
 * qgemm_moe_grouped: same arguments as qgemm_moe with perm in place of
 *   token_expert_idx; perm entries outside [0, T*topk) are skipped.
 */
int qgemm_moe_bucket(const int32_t* token_expert_idx, const int32_t* expert_offsets,
                     int32_t* perm, int n_assign, int E, hipStream_t stream);
int qgemm_moe_grouped(const void* x, const int32_t* perm, const int32_t* expert_offsets,
                      const void* const* wq, const void* const* scales, float* y,
                      int T, int E, int topk, int N, int K, int fmt, hipStream_t stream);

/*
 * Fused MoE gate/up projection with the SiLU-gated activation in its epilogue
 * (Section 3.1, fused gate/up item): for every assignment a routed to expert e
 * (perm and expert_offsets as for qgemm_moe_grouped) and i < inter,
 *   g = (dequant(wq[e], scales[e]) . x[a / topk])[i]
 *   u = (dequant(wq[e], scales[e]) . x[a / topk])[inter + i]
 *   h[a][i] = bf16_rne(silu(g) * u)
 * with g and u the same fp32 values qgemm_moe_grouped writes to y[a][i] and
 * y[a][inter + i], and silu evaluated as in qgemm_swiglu, so h equals
 * qgemm_swiglu applied to qgemm_moe_grouped's output bit for bit; the fp32
 * [T*topk][2*inter] intermediate is never stored.
 * wq[e], scales[e]: the gate rows (0 .. inter-1) and then the up rows
 * (inter .. 2*inter-1) of one [2*inter][K] matrix per expert, laid out as for
 * qgemm_dense with N = 2*inter; each matrix spans less than 4 GiB.
 * h: bf16 [T*topk][inter] in assignment order; rows of assignments absent
 * from perm are not written.
 * Sizes as for qgemm_moe with N = 2*inter, inter >= 1.
 */
int qgemm_moe_gate_up_swiglu(const void* x, const int32_t* perm, const int32_t* expert_offsets,
                             const void* const* wq, const void* const* scales, void* h,
                             int T, int E, int topk, int inter, int K, int fmt,
                             hipStream_t stream);

/*
 * MoE down projection with the router-weighted combine fused into it (the
 * MoE expert GEMM of Section 3.1 over the SiLU-gated activations, followed by
 * the weighted sum of each token's selected experts):
 *   y2[a][:] = dequant(wq[e], scales[e]) . h[a][:]        (a routed to expert e)
 *   out[t][n] = sum_{j < topk} route_w[t*topk + j] * y2[t*topk + j][n]
 * h: bf16 [T*topk][K], one row per token slot (as qgemm_moe_gate_up_swiglu
 * writes it); perm, expert_offsets: as for qgemm_moe_grouped over the T*topk
 * slots; wq, scales: HOST arrays of E device pointers, each [N][K] as for
 * qgemm_dense; route_w: fp32 [T*topk]; y2: fp32 [T*topk][N], caller-owned,
 * written with exactly the values qgemm_moe_grouped(h, perm, ..., topk = 1)
 * writes; out: fp32 [T][N], bitwise equal to qgemm_moe_combine(y2, route_w)
 * (each sum runs in increasing j from zero with fp32 fused multiply-adds).
 * The tile that stores the last of a token's topk slot rows for a column tile
 * sums them there, so the separate combine pass over y2 disappears; results
 * do not depend on which tile that is. Arrival counters live in a
 * library-owned workspace (grown on first use, freed by qgemm_release) and
 * are cleared by a kernel at the start of every call; calls that share it are
 * ordered only by their streams.
 * Sizes: as for qgemm_moe_grouped with T*topk rows; N % 4 == 0; y2 spans less
 * than 4 GiB (T*topk*N*4 bytes, else QGEMM_EUNSUPPORTED). Tokens whose slots
 * are not all present in perm (inconsistent routing tables) are not written.
 */
int qgemm_moe_down_combine(const void* h, const int32_t* perm, const int32_t* expert_offsets,
                           const void* const* wq, const void* const* scales, const float* route_w,
                           float* y2, float* out, int T, int E, int topk, int N, int K, int fmt,
                           hipStream_t stream);

/*
 * SiLU-gated activation between the MoE projections (Section 3.1, fused
 * gate/up item): for r < rows, i < inter,
 *   h[r][i] = bf16_rne(silu(y1[r][i]) * y1[r][inter + i]),  silu(z) = z / (1 + e^-z)
 * evaluated in fp32 with the hardware exponential and reciprocal (about one
 * fp32 ulp each, below the bf16 rounding of h).
 * y1: fp32 [rows][2*inter]; h: bf16 [rows][inter]. inter % 8 == 0.
 */
int qgemm_swiglu(const float* y1, void* h, int rows, int inter, hipStream_t stream);

/*
 * Router-weighted combine of the selected experts' outputs:
 *   out[t][n] = sum_{j < topk} route_w[t*topk + j] * y2[t*topk + j][n]
 * summed in increasing j in fp32. y2: fp32 [T*topk][N]; route_w: fp32
 * [T*topk]; out: fp32 [T][N]. N % 4 == 0.
 */
int qgemm_moe_combine(const float* y2, const float* route_w, float* out,
                      int T, int topk, int N, hipStream_t stream);

/* Message of the last non-OK return on the calling thread ("" if none). */
const char* qgemm_last_error(void);

/*
 * Prefill attention (Section 3.1, prefill attention item): softmax attention of a prompt's
 * queries over its keys, with the score product and the output product on the matrix cores and
 * an exact online softmax (running row maximum) between them. For every batch entry b, query
 * head h and query position i:
 *   s_j = scale * (q[b][i][h] . k[b][j][g]),  g = h / (H / Hkv)   (grouped-query attention)
 *   o[b][i][h] = sum_j softmax(s)_j v[b][j][g]
 * over the keys j <= i (causal = 1: prefill from an empty cache) or all keys j < S (causal = 0).
 * q, o: bf16 [B][S][H][D]; k, v: bf16 [B][S][Hkv][D]; every tensor contiguous, token-major,
 * 16-byte aligned; caller-owned device memory. D is 64 or 128; H a multiple of Hkv;
 * S*H*D < 2^31. Accumulation is fp32; the softmax weights enter the output product as bf16
 * and o is rounded to bf16 (nearest even). scale > 0 (1/sqrt(D) for the usual models).
 * Returns QGEMM_EINVAL / QGEMM_EUNSUPPORTED / QGEMM_EALIGN before launching anything (o is
 * untouched) and QGEMM_EHIP if the launch fails; B == 0 or S == 0 is a no-op.
 */
int qgemm_attention_prefill(const void* q, const void* k, const void* v, void* o,
                            int B, int S, int H, int Hkv, int D,
                            float scale, int causal, hipStream_t stream);

/*
 * Measurement utility, not part of the GEMM path: runs `iters` rounds of four
 * independent bf16 MFMAs (the GEMM's v_mfma_f32_32x32x16_bf16) in eight waves on
 * every CU at once, synchronises `stream`, and returns through HOST pointers
 * the median shader clock the CUs held (MHz; cycle counter over the device's
 * constant-rate real-time counter) and the bf16 dense matrix throughput the
 * launch reached (TFLOP/s, from HIP events on `stream`): the practical matrix-core
 * ceiling at the sustained clock, beside the nominal 2.4 GHz peak. Allocates and
 * frees its own small buffers. QGEMM_EINVAL for iters < 1 or null outputs.
 */
int qgemm_probe_mfma_clock(int iters, double* sclk_mhz, double* mfma_tflops, hipStream_t stream);

/* Frees the library-owned workspaces (MoE bucketing, split-K partials); the
 * next call that needs one grows it again. The caller must have synchronised
 * every stream that used them. */
int qgemm_release(void);

/* Library ABI version, (major << 16) | minor. */
int qgemm_version(void);

#ifdef __cplusplus
}
#endif

#endif /* QGEMM_H */
