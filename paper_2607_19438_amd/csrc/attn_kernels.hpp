// Prefill flash attention for gfx950 (Section 3.1, prefill attention item): the score product
// and the output product run on the matrix cores, with an exact online softmax (running row
// maximum, rescaling of the running output) between them.
//
// A workgroup (4 waves) owns 128 query rows of one (batch, query head); wave w owns rows
// 32w..32w+31. Keys and values stream through LDS in blocks of 64 (double-buffered, the next
// block's global loads in flight during the current block's math). Per block and wave:
//   S^T = K Q^T   (v_mfma_f32_32x32x16_bf16: keys as the A rows from LDS, the wave's queries as
//                  the B columns, held in registers for the whole loop) -- so each lane owns one
//                  query and 32 of the block's keys, and a row maximum needs one lane exchange;
//   online softmax on the scores in registers (exp2 with the scale folded into log2 e);
//   O^T += V^T P^T (the same MFMA: V^T read from the row-major value block with gfx950's
//                  transposing LDS read, P^T straight from the score registers rounded to bf16
//                  -- the score layout is the B-operand layout once the MFMA's 16-element K order
//                  is chosen to match it).
// Keys and values both go from HBM to LDS by DMA, with no register staging.
// Rows are normalised by the running sum at the end and stored as bf16. Causal blocks above the
// diagonal are skipped; blocks on it are masked key by key.
#pragma once

#include "qgemm_kernels.hpp"

namespace qg {

constexpr int kAttnThreads = 256;   // four waves
constexpr int kAttnBQ = 128;        // query rows per workgroup
constexpr int kAttnBK = 64;         // keys per block

struct AttnArgs {
  const uint16_t* q;   // bf16 [B][S][H][D]
  const uint16_t* k;   // bf16 [B][S][Hkv][D]
  const uint16_t* v;   // bf16 [B][S][Hkv][D]
  uint16_t* o;         // bf16 [B][S][H][D]
  int B;
  int S;
  int H;
  int Hkv;
  float sl2;           // softmax scale * log2(e)
};

// The kernel body lives in a device function (the kernel below only forwards to it): its
// scheduling builtins exist for the GPU target only, and a kernel template's host-side stub is
// not emitted when its own body uses them.
// The value of lane l ^ 32 (the other MFMA lane half of the same query), with one VALU lane swap.
__device__ __forceinline__ float other_half(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);   // {x[l % 32], x[32 + l % 32]}
  const int lane = (int)(threadIdx.x & 63);
  return __builtin_bit_cast(float, (unsigned)(lane < 32 ? r[1] : r[0]));
}

template <int D, bool CAUSAL>
__device__ __forceinline__ void attn_body(const AttnArgs& a) {
  static_assert(D == 64 || D == 128, "head dimension 64 or 128");
  constexpr int KCH = D / 8;                  // 16-byte chunks per key row
  constexpr int KSTEPS = D / 16;              // K16 steps of the score product
  constexpr int DT = D / 32;                  // 32-row tiles of O^T
  constexpr int KROWS_DMA = 1024 / (2 * D);   // key rows per 1 KiB DMA instruction
  constexpr int KDMA = kAttnBK / KROWS_DMA / 4;                 // key DMA instructions per wave
  // one __shared__ array per buffer, so the compiler can tell the key DMA into one buffer from
  // the LDS reads of the other and leaves the DMA in flight across them
  __shared__ __attribute__((aligned(16))) uint16_t ks0[kAttnBK * D];
  __shared__ __attribute__((aligned(16))) uint16_t ks1[kAttnBK * D];
  __shared__ __attribute__((aligned(16))) uint16_t vt0[kAttnBK * D];
  __shared__ __attribute__((aligned(16))) uint16_t vt1[kAttnBK * D];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31;     // this lane's query within the wave (MFMA column)
  const int hh = lane >> 5;      // MFMA lane half
  const int S = a.S, H = a.H;
  const int nqb = (S + kAttnBQ - 1) / kAttnBQ;
  int bh, qb;
  if (CAUSAL) {
    // heavy members (query blocks nqb-1 .. nqb-ceil(nqb/2)) of all heads first, then the light
    // members in the same order: workgroups L and L + (heavy count) are complementary
    const int hi = (nqb + 1) >> 1;
    const int lo = nqb >> 1;
    const int nh = a.B * H * hi;
    const int L = (int)blockIdx.x;
    if (L < nh) {
      bh = L / hi;
      qb = nqb - 1 - (L - bh * hi);
    } else {
      const int J = L - nh;
      bh = J / lo;
      qb = J - bh * lo;
    }
  } else {
    const int item = xcd_tile((int)blockIdx.x, a.B * H * nqb);
    bh = item / nqb;
    qb = item - bh * nqb;
  }
  const int b = bh / H;
  const int h = bh - b * H;
  const int g = h / (H / a.Hkv);
  const int q0 = qb * kAttnBQ;
  const int qrow = q0 + wave * 32 + col;      // this lane's query position

  const size_t qstride = (size_t)H * D;       // elements between consecutive tokens of q / o
  const size_t kstride = (size_t)a.Hkv * D;
  const __amdgpu_buffer_rsrc_t qr = make_rsrc(a.q + (size_t)b * S * qstride + (size_t)h * D,
                                              (uint32_t)(((size_t)(S - 1) * qstride + D) * 2));
  const __amdgpu_buffer_rsrc_t kr = make_rsrc(a.k + (size_t)b * S * kstride + (size_t)g * D,
                                              (uint32_t)(((size_t)(S - 1) * kstride + D) * 2));
  const __amdgpu_buffer_rsrc_t vr = make_rsrc(a.v + (size_t)b * S * kstride + (size_t)g * D,
                                              (uint32_t)(((size_t)(S - 1) * kstride + D) * 2));

  // query fragments (B operand of K Q^T): step t needs q[qrow][16t + 8hh .. +8]
  bf16x8 qf[KSTEPS];
#pragma unroll
  for (int t = 0; t < KSTEPS; ++t) {
    const uint32_t off = qrow < S ? ((uint32_t)qrow * (uint32_t)qstride + 16u * t + 8u * hh) * 2u : kOOB;
    qf[t] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(qr, off, 0, 0));
  }

  // 16-byte chunk swizzle of a key row in LDS: any 16 consecutive keys read at one logical chunk
  // hit 16 distinct bank groups, and any 8 hit 8 distinct 16-byte groups of a 128-byte bank
  // window (rows are 256 bytes at D = 128; at D = 64 the rows are 128 bytes, the layout of the
  // GEMM tiles, and take their row swizzle)
  auto kswz = [](int key) { return (D == 128) ? (key & 15) : row_swizzle(key); };
  // keys: DMA straight into LDS; lane L of a 1 KiB instruction fills physical chunk L % KCH of
  // key row L / KCH, so it fetches the logical chunk that the swizzle puts there
  const int dkey = lane / KCH;
  // per-lane byte offsets within a block (key row krow + dkey of the block; rows at or past S lie
  // beyond the end of the buffer range and read as zeros, so no per-block test is needed)
  uint32_t kdma_off[KDMA];
#pragma unroll
  for (int i = 0; i < KDMA; ++i) {
    const int krow = (wave * KDMA + i) * KROWS_DMA;
    kdma_off[i] = ((uint32_t)(krow + dkey) * (uint32_t)kstride + 8u * (uint32_t)((lane % KCH) ^ kswz(krow + dkey))) * 2u;
  }
  const uint32_t kblock_bytes = (uint32_t)kAttnBK * (uint32_t)kstride * 2u;   // one key block
  auto dma_keys = [&](uint16_t* ks, int jb) {
    const uint32_t base = (uint32_t)jb * kblock_bytes;
#pragma unroll
    for (int i = 0; i < KDMA; ++i) {
      const int krow = (wave * KDMA + i) * KROWS_DMA;          // first key row of this instruction
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (__attribute__((address_space(3))) void*)(ks + krow * D), 16,
                                               kdma_off[i] + base, 0, 0, 0);
    }
  };
  // values: DMA straight into LDS too, row-major (key rows), 16-byte chunks XOR-swizzled by
  // vswz(key); the output product reads them with the transposing LDS read, which hands each
  // lane 4 keys of one dimension. The swizzle puts the 4 consecutive keys x 64 bytes that the
  // 32 lanes of one half-wave read on 256 distinct bytes of the bank space.
  auto vswz = [](int key) { return (D == 128) ? 4 * (key & 3) : 4 * ((key >> 1) & 1); };
  uint32_t vdma_off[KDMA];
#pragma unroll
  for (int i = 0; i < KDMA; ++i) {
    const int krow = (wave * KDMA + i) * KROWS_DMA;
    vdma_off[i] = ((uint32_t)(krow + dkey) * (uint32_t)kstride + 8u * (uint32_t)((lane % KCH) ^ vswz(krow + dkey))) * 2u;
  }
  auto dma_values = [&](uint16_t* vs, int jb) {
    const uint32_t base = (uint32_t)jb * kblock_bytes;
#pragma unroll
    for (int i = 0; i < KDMA; ++i) {
      const int krow = (wave * KDMA + i) * KROWS_DMA;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (__attribute__((address_space(3))) void*)(vs + krow * D), 16,
                                               vdma_off[i] + base, 0, 0, 0);
    }
  };

  int nkb = (S + kAttnBK - 1) / kAttnBK;
  if (CAUSAL) nkb = min(nkb, (q0 + kAttnBQ - 1) / kAttnBK + 1);
  const int wq_last = q0 + wave * 32 + 31;    // the wave's last query row

  f32x16 acc_o[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i) acc_o[i] = f32x16{};
  float m_run = -__builtin_inff();   // running maximum of the raw scores q.k
  float l_run = 0.0f;
  const float sl2 = a.sl2;

  dma_keys(ks0, 0);
  dma_values(vt0, 0);
  wait_vmcnt_lgkm0<0>();
  __syncthreads();

  // LDS fragment reads: key rows (A operand of K Q^T) and transposed values (A operand of V^T P^T)
  auto rd_k = [&](const uint16_t* ksc, int t, int kt) {
    const int key = kt * 32 + col;
    const int c = 2 * t + hh;
    return *reinterpret_cast<const bf16x8*>(&ksc[key * D + ((c ^ kswz(key)) << 3)]);
  };
  // V^T fragment of MFMA step u, tile dt: lane (d = col, hh) needs the keys 16u + 4hh + {0..3}
  // and 16u + 8 + 4hh + {0..3} of dimension 32dt + col. In a transposing read each 16-lane group
  // returns, to lane i, element i % 4 of the 8-byte pieces that lanes 4r + i/4 (r = 0..3) point
  // at; so lane s of the group points at key (run start + s/4), dimensions 4(s%4)..+3 of the
  // group's 16, and lane i gets the run's 4 keys of dimension (group's first) + i.
  const int trk = (lane & 15) >> 2;                   // key within the run of 4
  const int trd = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);   // first of the 4 dims this lane points at
  auto rd_v = [&](const uint16_t* vtc, int u, int dt) {
    uint32_t w[4];
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int key = 16 * u + 8 * half + 4 * hh + trk;
      const int dim = 32 * dt + trd;
      const int e = key * D + (((dim >> 3) ^ vswz(key)) << 3) + (dim & 7);
      typedef short v4i16 __attribute__((ext_vector_type(4)));
      const v4i16 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) v4i16*)(const_cast<uint16_t*>(vtc) + e));
      const uint2 rr = __builtin_bit_cast(uint2, r);
      w[2 * half] = rr.x;
      w[2 * half + 1] = rr.y;
    }
    return __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
  };

  // one key block: math on buffer (ksc, vtc) while the next block's keys stream into (ksn, vtn)
  auto step = [&](int jb, const uint16_t* ksc, const uint16_t* vtc, uint16_t* ksn, uint16_t* vtn) {
    const int j0 = jb * kAttnBK;
    const bool more = jb + 1 < nkb;
    if (more) {
      dma_keys(ksn, jb + 1);
      dma_values(vtn, jb + 1);
    }
    if (!CAUSAL || j0 <= wq_last) {
      // scores S^T[key][query] for the block's 64 keys (two 32-key tiles, interleaved); the key
      // fragments of step t+2 are read from LDS while the MFMAs of step t run
      f32x16 sc[2] = {f32x16{}, f32x16{}};
      bf16x8 kf[3][2];
      kf[0][0] = rd_k(ksc, 0, 0);
      kf[0][1] = rd_k(ksc, 0, 1);
      kf[1][0] = rd_k(ksc, 1, 0);
      kf[1][1] = rd_k(ksc, 1, 1);
      // raised wave priority while a wave issues its MFMAs: the SIMD's other wave fills the
      // issue slots between them with its softmax VALU work
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int t = 0; t < KSTEPS; ++t) {
        if (t + 2 < KSTEPS) {
          kf[(t + 2) % 3][0] = rd_k(ksc, t + 2, 0);
          kf[(t + 2) % 3][1] = rd_k(ksc, t + 2, 1);
        }
        sc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[t % 3][0], qf[t], sc[0], 0, 0, 0);
        sc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[t % 3][1], qf[t], sc[1], 0, 0, 0);
        if (t + 2 < KSTEPS) QG_SG(kSchedDSRead, 2);
        QG_SG(kSchedMFMA, 2);
      }
      __builtin_amdgcn_s_setprio(0);
      // key of register r in tile kt: kt*32 + (r/4)*8 + 4hh + r%4
      const bool need_mask = (CAUSAL && j0 + kAttnBK - 1 > q0 + wave * 32) || j0 + kAttnBK > S;
      if (need_mask) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int kp = j0 + kt * 32 + (r >> 2) * 8 + 4 * hh + (r & 3);
            if (kp >= S || (CAUSAL && kp > qrow)) sc[kt][r] = -__builtin_inff();
          }
      }
      float mloc = -__builtin_inff();
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, sc[kt][r]);
      mloc = fmaxf(mloc, other_half(mloc));
      const float m_new = fmaxf(m_run, mloc);
      // The reference maximum m_run moves (and the running output and sum are rescaled, before
      // any of this block's output-product MFMAs) only when the block's maximum exceeds it by
      // more than 8 in exp2 units. Softmax does not depend on the reference as long as the
      // weights and their sum use the same one, and the threshold keeps every weight <= 2^8,
      // far inside fp32 and bf16 range; most blocks skip the rescale. (The first block always
      // moves it from -inf, with alpha = 0 on the empty sum.)
      if ((m_new - m_run) * sl2 > 8.0f) {
        const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * sl2);
        l_run *= alpha;
#pragma unroll
        for (int i = 0; i < DT; ++i) acc_o[i] *= alpha;
        m_run = m_new;
      }
      // p = exp2((s - m) * scale * log2 e), one fused multiply-add per score; P^T as packed bf16,
      // per key tile: registers (2i, 2i+1). Tile 1's exponentials are written between the
      // output-product MFMAs of tile 0 so the two overlap.
      const float ms = m_run * sl2;
      float lsum = 0.0f;
      uint32_t pf[2][8];
      auto exp_tile = [&](int kt) {
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[kt][r], sl2, -ms));
          const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[kt][r + 1], sl2, -ms));
          lsum += p0 + p1;
          pf[kt][r >> 1] = pack_bf16x2(p0, p1);
        }
      };
      exp_tile(0);
      // O^T += V^T P^T: K16 step u covers keys 16u..16u+15; lane half hh supplies the keys
      // 16u + 4hh + {0..3} and 16u + 8 + 4hh + {0..3} (its score registers 8(u%2)..8(u%2)+7).
      // The value fragments of step u+1 are read from LDS while the MFMAs of step u run.
      bf16x8 vf[2][DT];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) vf[0][dt] = rd_v(vtc, 0, dt);
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (u + 1 < 4) {
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) vf[(u + 1) & 1][dt] = rd_v(vtc, u + 1, dt);
        }
        const int kt = u >> 1;
        const int r0 = (u & 1) * 4;
        const bf16x8 pb = __builtin_bit_cast(bf16x8, u32x4{pf[kt][r0], pf[kt][r0 + 1], pf[kt][r0 + 2], pf[kt][r0 + 3]});
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          acc_o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[u & 1][dt], pb, acc_o[dt], 0, 0, 0);
        if (u == 0) exp_tile(1);
      }
      __builtin_amdgcn_s_setprio(0);
      l_run += lsum;
    }

    wait_vmcnt_lgkm0<0>();   // the key and value DMA of the next block are in LDS
    __syncthreads();
  };

  for (int jb = 0; jb < nkb; jb += 2) {
    step(jb, ks0, vt0, ks1, vt1);
    if (jb + 1 < nkb) step(jb + 1, ks1, vt1, ks0, vt0);
  }

  // normalise and store: lane (col, hh) holds o[qrow][dt*32 + 8a + 4hh + {0..3}] in acc_o[dt][4a..4a+3]
  const float l_tot = l_run + other_half(l_run);
  const float inv = 1.0f / l_tot;
  if (qrow < S) {
    uint16_t* orow = a.o + ((size_t)b * S + qrow) * qstride + (size_t)h * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int a4 = 0; a4 < 4; ++a4) {
        const uint32_t lo = pack_bf16x2(acc_o[dt][4 * a4] * inv, acc_o[dt][4 * a4 + 1] * inv);
        const uint32_t hi = pack_bf16x2(acc_o[dt][4 * a4 + 2] * inv, acc_o[dt][4 * a4 + 3] * inv);
        *reinterpret_cast<uint2*>(orow + dt * 32 + 8 * a4 + 4 * hh) = make_uint2(lo, hi);
      }
    }
  }
}

template <int D, bool CAUSAL>
__global__ __launch_bounds__(kAttnThreads, 2) void attn_fwd_kernel(AttnArgs a) {
  attn_body<D, CAUSAL>(a);
}

}  // namespace qg
