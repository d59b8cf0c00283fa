// Attention kernels for gfx950 (MI355X): bf16 inputs, fp32 accumulation on
// the matrix cores, fp32 online softmax in base 2.
//
// decode_gqa_kernel   decode phase, grouped-query heads (head dim 64 / 128):
//                     one work-group per (decode item, KV head); its waves take
//                     32-key chunks of the item's key range in turn, streaming
//                     K and V straight from HBM into registers.
// rowpar_kernel       prefill phase (all layouts) and decode of the 576/512
//                     latent layout: each wave owns 16 (or 32) query rows; the
//                     work-group stages key tiles, gathered through the block
//                     table, in double-buffered LDS shared by all waves.
//
// Both end in the flash-decoding merge when a decode sequence is split:
// every split writes (max, sum, unnormalised output) to the workspace and the
// last work-group of the (sequence, column) to arrive combines them in split
// order, so results are bit-identical run to run (no float atomics).
#include <math.h>

#include "device_common.h"
#include "kernels.h"

namespace flexattn {

__device__ __forceinline__ PagedCache as_cache(const CacheRef& c) { return PagedCache{c.base, c.sp, c.ss, c.sh}; }

// Combine the partials of splits first .. first+nspl-1 of one (sequence,
// column) and write bf16 rows out_row0 .. out_row0+rows-1 (and their lse).
template <int DV>
__device__ void merge_splits(const AttnParams& p, int first, int nspl, int col, int W, int rows,
                             int64_t out_row0, uint32_t* counter) {
  for (int idx = threadIdx.x; idx < rows * (DV / 2); idx += blockDim.x) {
    const int i = idx / (DV / 2);
    const int d = 2 * (idx % (DV / 2));
    float M = -INFINITY;
    for (int j = 0; j < nspl; ++j) {
      const int64_t slot = int64_t(first + j) * W + col;
      M = fmaxf(M, p.ws_stats[(slot * rows + i) * 2]);
    }
    float den = 0.f, o0 = 0.f, o1 = 0.f;
    for (int j = 0; j < nspl; ++j) {
      const int64_t slot = int64_t(first + j) * W + col;
      const float f = exp2f(p.ws_stats[(slot * rows + i) * 2] - M);
      den += f * p.ws_stats[(slot * rows + i) * 2 + 1];
      const float2 v = *reinterpret_cast<const float2*>(p.ws_o + (slot * rows + i) * DV + d);
      o0 += f * v.x;
      o1 += f * v.y;
    }
    const float inv = 1.f / den;
    *reinterpret_cast<uint32_t*>(p.out + (out_row0 + i) * DV + d) = pack_bf16x2(o0 * inv, o1 * inv);
    if (d == 0 && p.lse) p.lse[out_row0 + i] = (M + log2f(den)) * kLn2;
  }
  if (threadIdx.x == 0) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Publish this work-group's partial and report whether it arrived last.
__device__ __forceinline__ bool arrive_last(uint32_t* counter, int nspl) {
  __shared__ int s_last;
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    s_last = prev == uint32_t(nspl - 1);
  }
  __syncthreads();
  if (!s_last) return false;
  __threadfence();
  return true;
}

// ---------------------------------------------------------------------------
// Decode, grouped-query heads.
// ---------------------------------------------------------------------------
template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void decode_gqa_kernel(AttnParams p) {
  static_assert(D == 64 || D == 128, "head dim");
  constexpr int DC = D / 32;   // 32-dim chunks of the QK^T contraction
  constexpr int DPL = D / 16;  // value dims each lane owns in PV
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int n = lane & 15, gq = lane >> 4;
  const int item = blockIdx.x;
  const int g = blockIdx.y;
  const int W = gridDim.y;
  const int32_t* it = p.items + 8 * item;
  const int seq = it[0], nspl = it[2], k0 = it[3], first = it[5], dseq = it[6];
  const int L = p.seq_lens[seq];
  const int kend = min(it[4], L);
  const int tok = p.qsl[seq];
  const int32_t* bt_row = p.bt + int64_t(seq) * p.bt_stride;
  const int P = p.P;
  const int G = p.G;
  const PagedCache kc = as_cache(p.kc), vc = as_cache(p.vc);

  // Q as the B operand of S^T = K Q^T: column n = query head g*G + n.
  u32x4 qop[DC];
  {
    const bool ok = n < G;
    const uint16_t* qr = p.q + (int64_t(tok) * p.Hq + g * G + (ok ? n : 0)) * D;
#pragma unroll
    for (int c = 0; c < DC; ++c) qop[c] = ok ? load16(qr + 32 * c + 8 * gq) : zero4();
  }

  float m = -INFINITY, l = 0.f;
  f32x4 o[DPL];
#pragma unroll
  for (int a = 0; a < DPL; ++a) o[a] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nchunks = (kend - k0 + 31) >> 5;
  for (int ci = w; ci < nchunks; ci += NW) {
    const int kc0 = k0 + 32 * ci;
    const int page0 = page_of(bt_row, kc0, P);
    const int page1 = (kc0 + 16 < kend) ? page_of(bt_row, kc0 + 16, P) : page0;

    // K rows as the A operand: row n of block b is key kc0 + 16b + n.
    u32x4 kop[2][DC];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int key = kc0 + 16 * b + n;
      const bool ok = key < kend;
      const uint16_t* kr = kc.row(b ? page1 : page0, key % P, g);
#pragma unroll
      for (int c = 0; c < DC; ++c) kop[b][c] = ok ? load16(kr + 32 * c + 8 * gq) : zero4();
    }
    // V rows of the lane's 8 keys, value dims DPL*n .. DPL*n + DPL - 1.
    u32x4 vop[DPL];
    if constexpr (D == 128) {
      u32x4 rows[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int key = kc0 + chunk_key(e, gq);
        rows[e] = key < kend ? load16(vc.row((e >> 2) ? page1 : page0, key % P, g) + DPL * n) : zero4();
      }
      transpose8x8(rows, vop);
    } else {
      u32x2 rows[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int key = kc0 + chunk_key(e, gq);
        rows[e] = key < kend ? load8(vc.row((e >> 2) ? page1 : page0, key % P, g) + DPL * n) : u32x2{0u, 0u};
      }
      transpose8x4(rows, vop);
    }

    f32x4 s[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      s[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < DC; ++c) s[b] = mfma_16x16x32(kop[b][c], qop[c], s[b]);
    }

    // Online softmax for query row n over the chunk's keys (base 2).
    float z[8];
    float cmax = -INFINITY;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int key = kc0 + chunk_key(e, gq);
      z[e] = key < kend ? s[e >> 2][e & 3] * p.scale_log2 : -INFINITY;
      cmax = fmaxf(cmax, z[e]);
    }
    cmax = group_max(cmax);
    const float m_new = fmaxf(m, cmax);
    const float alpha = exp2f(m - m_new);
    u32x4 pop;
    float psum = 0.f;
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      const float p0 = exp2f(z[2 * e2] - m_new);
      const float p1 = exp2f(z[2 * e2 + 1] - m_new);
      psum += p0 + p1;
      pop[e2] = pack_bf16x2(p0, p1);
    }
    l = l * alpha + psum;
    m = m_new;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float ar = shfl_f(alpha, 4 * gq + r);
#pragma unroll
      for (int a = 0; a < DPL; ++a) o[a][r] *= ar;
    }
#pragma unroll
    for (int a = 0; a < DPL; ++a) o[a] = mfma_16x16x32(pop, vop[a], o[a]);
  }

  // Combine the waves' partial states through LDS.
  const float ltot = group_sum(l);
  __shared__ float s_m[NW][16];
  __shared__ float s_l[NW][16];
  __shared__ float s_o[NW][16][D];
  if (gq == 0) {
    s_m[w][n] = m;
    s_l[w][n] = ltot;
  }
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int a = 0; a < DPL; ++a) s_o[w][4 * gq + r][DPL * n + a] = o[a][r];
  __syncthreads();

  const bool single = nspl == 1;
  const int64_t out_row0 = int64_t(tok) * p.Hq + int64_t(g) * G;
  const int64_t slot = int64_t(item) * W + g;
  for (int idx = threadIdx.x; idx < G * (D / 2); idx += NW * 64) {
    const int i = idx / (D / 2), d = 2 * (idx % (D / 2));
    float M = s_m[0][i];
#pragma unroll
    for (int ww = 1; ww < NW; ++ww) M = fmaxf(M, s_m[ww][i]);
    float den = 0.f, o0 = 0.f, o1 = 0.f;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) {
      const float f = exp2f(s_m[ww][i] - M);
      den += f * s_l[ww][i];
      o0 += f * s_o[ww][i][d];
      o1 += f * s_o[ww][i][d + 1];
    }
    if (single) {
      const float inv = 1.f / den;
      *reinterpret_cast<uint32_t*>(p.out + (out_row0 + i) * D + d) = pack_bf16x2(o0 * inv, o1 * inv);
      if (d == 0 && p.lse) p.lse[out_row0 + i] = (M + log2f(den)) * kLn2;
    } else {
      *reinterpret_cast<float2*>(p.ws_o + (slot * p.rows_per_wg + i) * D + d) = make_float2(o0, o1);
      if (d == 0) {
        p.ws_stats[(slot * p.rows_per_wg + i) * 2] = M;
        p.ws_stats[(slot * p.rows_per_wg + i) * 2 + 1] = den;
      }
    }
  }
  if (single) return;
  uint32_t* counter = p.counters + int64_t(dseq) * W + g;
  if (!arrive_last(counter, nspl)) return;
  merge_splits<D>(p, first, nspl, g, W, p.rows_per_wg, out_row0, counter);
}

// ---------------------------------------------------------------------------
// Row-parallel attention: prefill (GQA and latent) and latent decode.
// ---------------------------------------------------------------------------
template <int DQK, int DV, int NW, int RB, int BN, bool VALIAS, bool DECODE>
struct RowParCfg {
  static constexpr int DC = DQK / 32;
  static constexpr int LDS_ROW = DQK + 8;                 // 16-byte pad per row
  static constexpr int LDS_ROW_V = VALIAS ? LDS_ROW : DV + 8;
  static constexpr int CPR = DQK / 8;                     // 16-byte chunks per K row
  static constexpr int CPRV = VALIAS ? 0 : DV / 8;
  static constexpr int NT = NW * 64;
  static constexpr int TILE_CHUNKS = BN * (CPR + CPRV);
  static constexpr int NLD = TILE_CHUNKS / NT;
  static constexpr int NACC = DV / 16;
  static constexpr int NVG = DV >= 128 ? DV / 128 : 1;   // value-dim groups of 8 per lane
  static constexpr int K_ELEMS = BN * LDS_ROW;
  static constexpr int V_ELEMS = VALIAS ? 0 : BN * LDS_ROW_V;
  static constexpr size_t LDS_BYTES = size_t(2) * (K_ELEMS + V_ELEMS) * 2;
  static_assert(TILE_CHUNKS % NT == 0, "tile chunks must divide evenly");
  static_assert((BN * CPR) % NT == 0, "K chunks must divide evenly");
  static_assert(BN % 32 == 0, "key tile is a multiple of 32");
};

template <int DQK, int DV, int NW, int RB, int BN, bool VALIAS, bool DECODE>
__global__ __launch_bounds__(NW * 64) void rowpar_kernel(AttnParams p) {
  using C = RowParCfg<DQK, DV, NW, RB, BN, VALIAS, DECODE>;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  uint16_t* ldsK = lds;
  uint16_t* ldsV = VALIAS ? lds : lds + 2 * C::K_ELEMS;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int n = lane & 15, gq = lane >> 4;
  const int32_t* it = p.items + 8 * blockIdx.x;
  const int seq = it[0];
  const int L = p.seq_lens[seq];
  const int q0 = p.qsl[seq];
  const int nq = p.qsl[seq + 1] - q0;
  const int32_t* bt_row = p.bt + int64_t(seq) * p.bt_stride;
  const int P = p.P;
  const PagedCache kc = as_cache(p.kc), vc = as_cache(p.vc);

  int key_begin, key_end, head_kv, wave_limit;
  int row_tok[RB], row_head[RB], row_limit[RB];
  if constexpr (DECODE) {
    key_begin = it[3];
    key_end = min(it[4], L);
    const int hg = blockIdx.y;
    head_kv = (hg * p.rows_per_wg) / p.G;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      row_tok[rb] = q0;
      row_head[rb] = hg * p.rows_per_wg + (w * RB + rb) * 16 + n;
      row_limit[rb] = key_end;
    }
    wave_limit = key_end;
  } else {
    const int r0 = it[2], r1 = it[3];
    key_begin = 0;
    key_end = it[4];
    const int h = blockIdx.y;
    head_kv = h / p.G;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int local = r0 + (w * RB + rb) * 16 + n;
      const bool ok = local < r1;
      row_tok[rb] = q0 + (ok ? local : r0);
      row_head[rb] = h;
      row_limit[rb] = ok ? (L - nq + local + 1) : 1;
    }
    const int last = min(r1, r0 + (w + 1) * RB * 16) - 1;
    wave_limit = (r0 + w * RB * 16 < r1) ? (L - nq + last + 1) : 0;
  }

  // Q as the B operand of S^T = K Q^T.
  u32x4 qop[RB][C::DC];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const uint16_t* qr = p.q + (int64_t(row_tok[rb]) * p.Hq + row_head[rb]) * DQK;
#pragma unroll
    for (int c = 0; c < C::DC; ++c) qop[rb][c] = load16(qr + 32 * c + 8 * gq);
  }

  float m[RB], l[RB];
  f32x4 o[RB][C::NACC];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m[rb] = -INFINITY;
    l[rb] = 0.f;
#pragma unroll
    for (int a = 0; a < C::NACC; ++a) o[rb][a] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int ntiles = (key_end - key_begin + BN - 1) / BN;
  u32x4 stage[C::NLD];

  // Gather one key tile (keys kb .. kb+BN-1) through the block table into registers.
  auto load_tile = [&](int kb) {
#pragma unroll
    for (int i = 0; i < C::NLD; ++i) {
      const int u = i * C::NT + tid;
      if (u < BN * C::CPR) {
        const int r = u / C::CPR, x = u % C::CPR;
        const int key = kb + r;
        stage[i] = key < key_end ? load16(kc.row(page_of(bt_row, key, P), key % P, head_kv) + 8 * x) : zero4();
      } else {
        const int u2 = u - BN * C::CPR;
        const int r = u2 / (C::CPRV > 0 ? C::CPRV : 1), x = u2 % (C::CPRV > 0 ? C::CPRV : 1);
        const int key = kb + r;
        stage[i] = key < key_end ? load16(vc.row(page_of(bt_row, key, P), key % P, head_kv) + 8 * x) : zero4();
      }
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < C::NLD; ++i) {
      const int u = i * C::NT + tid;
      if (u < BN * C::CPR) {
        const int r = u / C::CPR, x = u % C::CPR;
        *reinterpret_cast<u32x4*>(ldsK + buf * C::K_ELEMS + r * C::LDS_ROW + 8 * x) = stage[i];
      } else {
        const int u2 = u - BN * C::CPR;
        const int r = u2 / (C::CPRV > 0 ? C::CPRV : 1), x = u2 % (C::CPRV > 0 ? C::CPRV : 1);
        *reinterpret_cast<u32x4*>(ldsV + buf * C::V_ELEMS + r * C::LDS_ROW_V + 8 * x) = stage[i];
      }
    }
  };

  if (ntiles > 0) {
    load_tile(key_begin);
    store_tile(0);
  }
  __syncthreads();

  for (int kt = 0; kt < ntiles; ++kt) {
    const int kb = key_begin + kt * BN;
    const int buf = kt & 1;
    if (kt + 1 < ntiles) load_tile(kb + BN);
    const uint16_t* Kt = ldsK + buf * C::K_ELEMS;
    const uint16_t* Vt = VALIAS ? Kt : ldsV + buf * C::V_ELEMS;

#pragma unroll
    for (int ch = 0; ch < BN / 32; ++ch) {
      const int kc0 = kb + 32 * ch;
      if (kc0 >= wave_limit) break;
      f32x4 s[RB][2];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) s[rb][0] = s[rb][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const uint16_t* kr = Kt + (32 * ch + 16 * b + n) * C::LDS_ROW + 8 * gq;
#pragma unroll
        for (int c = 0; c < C::DC; ++c) {
          const u32x4 kop = *reinterpret_cast<const u32x4*>(kr + 32 * c);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) s[rb][b] = mfma_16x16x32(kop, qop[rb][c], s[rb][b]);
        }
      }
      u32x4 pop[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        float z[8];
        float cmax = -INFINITY;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int key = kc0 + chunk_key(e, gq);
          z[e] = key < row_limit[rb] ? s[rb][e >> 2][e & 3] * p.scale_log2 : -INFINITY;
          cmax = fmaxf(cmax, z[e]);
        }
        cmax = group_max(cmax);
        const float m_new = fmaxf(m[rb], cmax);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = exp2f(m[rb] - m_use);
        float psum = 0.f;
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          const float p0 = exp2f(z[2 * e2] - m_use);
          const float p1 = exp2f(z[2 * e2 + 1] - m_use);
          psum += p0 + p1;
          pop[rb][e2] = pack_bf16x2(p0, p1);
        }
        l[rb] = l[rb] * alpha + psum;
        m[rb] = m_new;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float ar = shfl_f(alpha, 4 * gq + r);
#pragma unroll
          for (int a = 0; a < C::NACC; ++a) o[rb][a][r] *= ar;
        }
      }
      // PV: lane reads its 8 keys' value dims and transposes them in registers.
#pragma unroll
      for (int vg = 0; vg < C::NVG; ++vg) {
        if constexpr (DV >= 128) {
          u32x4 rows[8], vop[8];
#pragma unroll
          for (int e = 0; e < 8; ++e)
            rows[e] = *reinterpret_cast<const u32x4*>(Vt + (32 * ch + chunk_key(e, gq)) * C::LDS_ROW_V + 128 * vg + 8 * n);
          transpose8x8(rows, vop);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int c = 0; c < 8; ++c) o[rb][8 * vg + c] = mfma_16x16x32(pop[rb], vop[c], o[rb][8 * vg + c]);
        } else {
          u32x2 rows[8];
          u32x4 vop[4];
#pragma unroll
          for (int e = 0; e < 8; ++e)
            rows[e] = *reinterpret_cast<const u32x2*>(Vt + (32 * ch + chunk_key(e, gq)) * C::LDS_ROW_V + 4 * n);
          transpose8x4(rows, vop);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int c = 0; c < 4; ++c) o[rb][c] = mfma_16x16x32(pop[rb], vop[c], o[rb][c]);
        }
      }
    }

    if (kt + 1 < ntiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  // Epilogue. Lane (n, gq) holds output rows 4*gq + r of each row block, at
  // value dims 128*vg + 8*n + c (DV >= 128) or 4*n + c (DV = 64).
  auto row_values = [&](int rb, int r, float scale, uint16_t* dst_row) {
    if constexpr (DV >= 128) {
#pragma unroll
      for (int vg = 0; vg < C::NVG; ++vg) {
        u32x4 pk;
#pragma unroll
        for (int c2 = 0; c2 < 4; ++c2)
          pk[c2] = pack_bf16x2(o[rb][8 * vg + 2 * c2][r] * scale, o[rb][8 * vg + 2 * c2 + 1][r] * scale);
        *reinterpret_cast<u32x4*>(dst_row + 128 * vg + 8 * n) = pk;
      }
    } else {
      u32x2 pk;
      pk[0] = pack_bf16x2(o[rb][0][r] * scale, o[rb][1][r] * scale);
      pk[1] = pack_bf16x2(o[rb][2][r] * scale, o[rb][3][r] * scale);
      *reinterpret_cast<u32x2*>(dst_row + 4 * n) = pk;
    }
  };

  if constexpr (!DECODE) {
    const int r0 = it[2], r1 = it[3];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const float lt = group_sum(l[rb]);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rowi = (w * RB + rb) * 16 + 4 * gq + r;
        const float lr = shfl_f(lt, 4 * gq + r);
        const int local = r0 + rowi;
        if (local < r1) {
          const int64_t orow = int64_t(q0 + local) * p.Hq + row_head[rb];
          row_values(rb, r, 1.f / lr, p.out + orow * DV);
        }
      }
      const int local = r0 + (w * RB + rb) * 16 + n;
      if (gq == 0 && local < r1 && p.lse)
        p.lse[int64_t(q0 + local) * p.Hq + row_head[rb]] = (m[rb] + log2f(lt)) * kLn2;
    }
  } else {
    const int nspl = it[2], first = it[5], dseq = it[6];
    const int hg = blockIdx.y;
    const int W = gridDim.y;
    const int rows = p.rows_per_wg;
    const int64_t out_row0 = int64_t(q0) * p.Hq + int64_t(hg) * rows;
    const int64_t slot = int64_t(blockIdx.x) * W + hg;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const float lt = group_sum(l[rb]);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rowi = (w * RB + rb) * 16 + 4 * gq + r;
        const float lr = shfl_f(lt, 4 * gq + r);
        if (nspl == 1) {
          row_values(rb, r, 1.f / lr, p.out + (out_row0 + rowi) * DV);
        } else {
          float* dst = p.ws_o + (slot * rows + rowi) * DV;
          if constexpr (DV >= 128) {
#pragma unroll
            for (int vg = 0; vg < C::NVG; ++vg) {
              f32x4 a0, a1;
#pragma unroll
              for (int c = 0; c < 4; ++c) {
                a0[c] = o[rb][8 * vg + c][r];
                a1[c] = o[rb][8 * vg + 4 + c][r];
              }
              *reinterpret_cast<f32x4*>(dst + 128 * vg + 8 * n) = a0;
              *reinterpret_cast<f32x4*>(dst + 128 * vg + 8 * n + 4) = a1;
            }
          } else {
            f32x4 a0;
#pragma unroll
            for (int c = 0; c < 4; ++c) a0[c] = o[rb][c][r];
            *reinterpret_cast<f32x4*>(dst + 4 * n) = a0;
          }
        }
      }
      const int rown = (w * RB + rb) * 16 + n;
      if (gq == 0) {
        if (nspl == 1) {
          if (p.lse) p.lse[out_row0 + rown] = (m[rb] + log2f(lt)) * kLn2;
        } else {
          p.ws_stats[(slot * rows + rown) * 2] = m[rb];
          p.ws_stats[(slot * rows + rown) * 2 + 1] = lt;
        }
      }
    }
    if (nspl == 1) return;
    uint32_t* counter = p.counters + int64_t(dseq) * W + hg;
    if (!arrive_last(counter, nspl)) return;
    merge_splits<DV>(p, first, nspl, hg, W, rows, out_row0, counter);
  }
}

// ---------------------------------------------------------------------------
// Test aid: gather one sequence's rows through the same page arithmetic.
// ---------------------------------------------------------------------------
__global__ void gather_kernel(CacheRef kref, CacheRef vref, int has_v, const int32_t* bt_row, int32_t L,
                              int32_t P, int32_t Hkv, int32_t dqk, int32_t dv, uint16_t* k_out,
                              uint16_t* v_out) {
  const PagedCache kc = as_cache(kref), vc = as_cache(vref);
  const int64_t total = int64_t(L) * Hkv;
  for (int64_t r = blockIdx.x * int64_t(blockDim.y) + threadIdx.y; r < total; r += int64_t(gridDim.x) * blockDim.y) {
    const int t = int(r / Hkv), h = int(r % Hkv);
    const int page = page_of(bt_row, t, P);
    const uint16_t* ks = kc.row(page, t % P, h);
    for (int d = threadIdx.x; d < dqk; d += blockDim.x) k_out[r * dqk + d] = ks[d];
    if (has_v) {
      const uint16_t* vs = vc.row(page, t % P, h);
      for (int d = threadIdx.x; d < dv; d += blockDim.x) v_out[r * dv + d] = vs[d];
    }
  }
}

__global__ void fill_zero_kernel(uint32_t* p, size_t words) {
  for (size_t i = blockIdx.x * size_t(blockDim.x) + threadIdx.x; i < words; i += size_t(gridDim.x) * blockDim.x)
    p[i] = 0u;
}

// ---------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------
template <int DQK, int DV, int NW, int RB, int BN, bool VALIAS, bool DECODE>
static hipError_t launch_rowpar(const AttnParams& p, dim3 grid, hipStream_t stream) {
  using C = RowParCfg<DQK, DV, NW, RB, BN, VALIAS, DECODE>;
  auto kern = rowpar_kernel<DQK, DV, NW, RB, BN, VALIAS, DECODE>;
  static hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, int(C::LDS_BYTES));
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kern, grid, dim3(C::NT), C::LDS_BYTES, stream, p);
  return hipGetLastError();
}

hipError_t launch_decode(const AttnParams& p, int dqk, hipStream_t stream) {
  if (p.n_items == 0) return hipSuccess;
  const dim3 grid(p.n_items, p.grid_y);
  switch (dqk) {
    case 128:
      hipLaunchKernelGGL((decode_gqa_kernel<128, 4>), grid, dim3(256), 0, stream, p);
      return hipGetLastError();
    case 64:
      hipLaunchKernelGGL((decode_gqa_kernel<64, 4>), grid, dim3(256), 0, stream, p);
      return hipGetLastError();
    case 576:
      return launch_rowpar<576, 512, 4, 1, 32, true, true>(p, grid, stream);
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_prefill(const AttnParams& p, int dqk, int bm, hipStream_t stream) {
  if (p.n_items == 0) return hipSuccess;
  const dim3 grid(p.n_items, p.grid_y);
  if (dqk == 128 && bm == 128) return launch_rowpar<128, 128, 4, 2, 64, false, false>(p, grid, stream);
  if (dqk == 128 && bm == 64) return launch_rowpar<128, 128, 4, 1, 64, false, false>(p, grid, stream);
  if (dqk == 64 && bm == 128) return launch_rowpar<64, 64, 4, 2, 64, false, false>(p, grid, stream);
  if (dqk == 64 && bm == 64) return launch_rowpar<64, 64, 4, 1, 64, false, false>(p, grid, stream);
  if (dqk == 576 && bm == 64) return launch_rowpar<576, 512, 4, 1, 32, true, false>(p, grid, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_gather(const CacheRef& kc, const CacheRef& vc, bool has_v, const int32_t* bt_row, int32_t L,
                         int32_t P, int32_t Hkv, int32_t dqk, int32_t dv, uint16_t* k_out, uint16_t* v_out,
                         hipStream_t stream) {
  if (L == 0) return hipSuccess;
  const int64_t rows = int64_t(L) * Hkv;
  const int blocks = int(std::min<int64_t>((rows + 3) / 4, 4096));
  hipLaunchKernelGGL(gather_kernel, dim3(blocks), dim3(64, 4), 0, stream, kc, vc, has_v ? 1 : 0, bt_row, L, P,
                     Hkv, dqk, dv, k_out, v_out);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream) {
  const size_t words = bytes / 4;
  if (words == 0) return hipSuccess;
  const int blocks = int(std::min<size_t>((words + 255) / 256, 2048));
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, stream, static_cast<uint32_t*>(ptr), words);
  return hipGetLastError();
}

}  // namespace flexattn
