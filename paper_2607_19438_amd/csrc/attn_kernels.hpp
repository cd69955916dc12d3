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
//   O^T += V^T P^T (the same MFMA: V^T from an LDS copy of the value block transposed at write
//                  time, P^T straight from the score registers rounded to bf16 -- the score
//                  layout is the B-operand layout once the MFMA's 16-element K order is chosen
//                  to match it).
// Rows are normalised by the running sum at the end and stored as bf16. Causal blocks above the
// diagonal are skipped; blocks on it are masked key by key.
#pragma once

#include "qgemm_kernels.hpp"

namespace qg {

constexpr int kAttnThreads = 256;   // four waves
constexpr int kAttnBQ = 128;        // query rows per workgroup
constexpr int kAttnBK = 64;         // keys per block
constexpr int kAttnVPad = 4;        // bf16 padding of a transposed-value LDS row (bank spread)

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

template <int D, bool CAUSAL>
__global__ __launch_bounds__(kAttnThreads, 2) void attn_fwd_kernel(AttnArgs a) {
  static_assert(D == 64 || D == 128, "head dimension 64 or 128");
  constexpr int KCH = D / 8;                  // 16-byte chunks per key row
  constexpr int KSTEPS = D / 16;              // K16 steps of the score product
  constexpr int DT = D / 32;                  // 32-row tiles of O^T
  constexpr int VROW = kAttnBK + kAttnVPad;   // bf16 per transposed-value row
  constexpr int KLOADS = kAttnBK * KCH / kAttnThreads;          // 16-byte key loads per thread
  constexpr int VITEMS = (kAttnBK / 4) * (D / 8);               // (4 keys x 8 dims) value items
  __shared__ __attribute__((aligned(16))) uint16_t ks[2][kAttnBK * D];
  __shared__ __attribute__((aligned(16))) uint16_t vt[2][D * VROW];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int col = lane & 31;     // this lane's query within the wave (MFMA column)
  const int hh = lane >> 5;      // MFMA lane half
  const int S = a.S, H = a.H;
  const int nqb = (S + kAttnBQ - 1) / kAttnBQ;
  const int total = a.B * H * nqb;
  // XCD-grouped order: each XCD takes a contiguous range (heads of one key/value group), and
  // inside a head the query blocks with the most keys come first
  const int item = xcd_tile((int)blockIdx.x, total);
  const int bh = item / nqb;
  const int qb = nqb - 1 - (item - bh * nqb);
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
  // hit 16 distinct bank groups (rows are 256 bytes at D = 128, two rows share 256 bytes at 64)
  auto kswz = [](int key) { return (D == 128) ? (key & 15) : ((key >> 1) & 7); };
  // global -> registers for one key/value block
  uint4 kreg[KLOADS];
  uint4 vreg[4];
  const bool vitem = tid < VITEMS;
  const int vkg = tid / (D / 8);               // value item: keys 4vkg..4vkg+3
  const int vdg = tid - vkg * (D / 8);         //             dims 8vdg..8vdg+7
  auto load_block = [&](int j0) {
#pragma unroll
    for (int i = 0; i < KLOADS; ++i) {
      const int idx = tid + i * kAttnThreads;
      const int key = idx / KCH;
      const int c = idx - key * KCH;
      const int kp = j0 + key;
      const uint32_t off = kp < S ? ((uint32_t)kp * (uint32_t)kstride + 8u * c) * 2u : kOOB;
      kreg[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(kr, off, 0, 0));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int kp = j0 + 4 * vkg + i;
      const uint32_t off = (vitem && kp < S) ? ((uint32_t)kp * (uint32_t)kstride + 8u * vdg) * 2u : kOOB;
      vreg[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(vr, off, 0, 0));
    }
  };
  // registers -> LDS buffer `buf`: keys row-major with swizzled 16-byte chunks, values
  // transposed (row = dimension, 4 consecutive keys per 8-byte write)
  auto store_block = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KLOADS; ++i) {
      const int idx = tid + i * kAttnThreads;
      const int key = idx / KCH;
      const int c = idx - key * KCH;
      *reinterpret_cast<uint4*>(&ks[buf][key * D + ((c ^ kswz(key)) << 3)]) = kreg[i];
    }
    if (vitem) {
      const uint32_t w0[4] = {vreg[0].x, vreg[0].y, vreg[0].z, vreg[0].w};
      const uint32_t w1[4] = {vreg[1].x, vreg[1].y, vreg[1].z, vreg[1].w};
      const uint32_t w2[4] = {vreg[2].x, vreg[2].y, vreg[2].z, vreg[2].w};
      const uint32_t w3[4] = {vreg[3].x, vreg[3].y, vreg[3].z, vreg[3].w};
#pragma unroll
      for (int w = 0; w < 4; ++w) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const uint32_t sel = e ? 0x07060302u : 0x05040100u;   // high or low halves of two dwords
          const uint32_t lo = __builtin_amdgcn_perm(w1[w], w0[w], sel);
          const uint32_t hi = __builtin_amdgcn_perm(w3[w], w2[w], sel);
          const int d = 8 * vdg + 2 * w + e;
          *reinterpret_cast<uint2*>(&vt[buf][d * VROW + 4 * vkg]) = make_uint2(lo, hi);
        }
      }
    }
  };

  int nkb = (S + kAttnBK - 1) / kAttnBK;
  if (CAUSAL) nkb = min(nkb, (q0 + kAttnBQ - 1) / kAttnBK + 1);
  const int wq_last = q0 + wave * 32 + 31;    // the wave's last query row

  f32x16 acc_o[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i) acc_o[i] = f32x16{};
  float m_run = -__builtin_inff();
  float l_run = 0.0f;

  load_block(0);
  store_block(0);
  __syncthreads();

  for (int jb = 0; jb < nkb; ++jb) {
    const int cur = jb & 1;
    const int j0 = jb * kAttnBK;
    if (jb + 1 < nkb) load_block(j0 + kAttnBK);

    if (!CAUSAL || j0 <= wq_last) {
      // scores S^T[key][query] for the block's 64 keys (two 32-key tiles)
      f32x16 sc[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const int key = kt * 32 + col;
#pragma unroll
        for (int t = 0; t < KSTEPS; ++t) {
          const int c = 2 * t + hh;
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&ks[cur][key * D + ((c ^ kswz(key)) << 3)]);
          sc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[t], sc[kt], 0, 0, 0);
        }
      }
      // key of register r in tile kt: kt*32 + (r/4)*8 + 4hh + r%4
      const bool need_mask = (CAUSAL && j0 + kAttnBK - 1 > q0 + wave * 32) || j0 + kAttnBK > S;
      float mloc = -__builtin_inff();
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float x = sc[kt][r] * a.sl2;
          if (need_mask) {
            const int kp = j0 + kt * 32 + (r >> 2) * 8 + 4 * hh + (r & 3);
            if (kp >= S || (CAUSAL && kp > qrow)) x = -__builtin_inff();
          }
          sc[kt][r] = x;
          mloc = fmaxf(mloc, x);
        }
      }
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
      const float m_new = fmaxf(m_run, mloc);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      float lsum = 0.0f;
      uint32_t pf[2][8];   // P^T as packed bf16, per key tile: registers (2i, 2i+1)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const float p0 = __builtin_amdgcn_exp2f(sc[kt][r] - m_new);
          const float p1 = __builtin_amdgcn_exp2f(sc[kt][r + 1] - m_new);
          lsum += p0 + p1;
          pf[kt][r >> 1] = pack_bf16x2(p0, p1);
        }
      }
      l_run = l_run * alpha + lsum;
#pragma unroll
      for (int i = 0; i < DT; ++i) acc_o[i] *= alpha;
      // O^T += V^T P^T: K16 step u covers keys 16u..16u+15; lane half hh supplies the keys
      // 16u + 4hh + {0..3} and 16u + 8 + 4hh + {0..3} (its score registers 8(u%2)..8(u%2)+7)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int kt = u >> 1;
        const int r0 = (u & 1) * 4;
        const bf16x8 pb = __builtin_bit_cast(bf16x8, u32x4{pf[kt][r0], pf[kt][r0 + 1], pf[kt][r0 + 2], pf[kt][r0 + 3]});
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const uint16_t* row = &vt[cur][(dt * 32 + col) * VROW + 16 * u + 4 * hh];
          const uint2 lo = *reinterpret_cast<const uint2*>(row);
          const uint2 hi = *reinterpret_cast<const uint2*>(row + 8);
          const bf16x8 vf = __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, hi.x, hi.y});
          acc_o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb, acc_o[dt], 0, 0, 0);
        }
      }
    }

    if (jb + 1 < nkb) store_block(cur ^ 1);
    __syncthreads();
  }

  // normalise and store: lane (col, hh) holds o[qrow][dt*32 + 8a + 4hh + {0..3}] in acc_o[dt][4a..4a+3]
  const float l_tot = l_run + __shfl_xor(l_run, 32);
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

}  // namespace qg
