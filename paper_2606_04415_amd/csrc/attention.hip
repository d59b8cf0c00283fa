// Attention kernels for gfx950 (MI355X): bf16 inputs, fp32 accumulation on
// the matrix cores, fp32 online softmax in base 2.
//
// decode_gqa_kernel   decode phase, grouped-query heads (head dim 64 / 128):
//                     one work-group per (decode item, KV head); its waves take
//                     32-key chunks of the item's key range in turn, streaming
//                     K and V from HBM into registers (K through a wave-private
//                     LDS buffer that turns whole-line loads into MFMA rows).
// rowpar_kernel       prefill phase (all layouts) and decode of the 576/512
//                     latent layout: each wave owns 16 or 32 query rows; the
//                     work-group streams key tiles, gathered through the block
//                     table, into a ring of LDS stages shared by all waves.
//                     flat_prefill_kernel (grouped-query rows of one KV head)
//                     and perhead_prefill_kernel (heads split out) run the
//                     same body with their own register budgets.
// merge_kernel        flash-decoding combine of a split decode sequence: every
//                     split writes (max, sum, unnormalised output) to the
//                     workspace; a second launch combines them in split order,
//                     so results are bit-identical run to run (no float
//                     atomics).
#include <float.h>
#include <math.h>

#include <mutex>
#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace flexattn {

__device__ __forceinline__ PagedCache as_cache(const CacheRef& c) { return PagedCache{c.base, c.sp, c.ss, c.sh}; }

// Split-K merge (flash-decoding combine), one work-group per (decode piece,
// column); only piece 0 of a split sequence does work. Runs as its own launch
// after the decode kernel, so every partial is visible without device-scope
// fences. Each thread owns 4 value columns of one row and folds the pieces in
// ascending order, 8 at a time with all their loads in flight, keeping a
// running maximum M: results are bit-identical run to run. The result is
//   out = sum_j 2^{m_j - M} O_j / sum_j 2^{m_j - M} l_j,
//   lse = (M + log2 sum_j 2^{m_j - M} l_j) * ln 2     (m_j in log2 units).
template <int DV>
__global__ __launch_bounds__(256) void merge_kernel(AttnParams p) {
  constexpr int KB = 8;   // pieces folded per step
  const int32_t* it = p.items + 8 * p.merge[blockIdx.x];   // the sequence's first piece
  const int slot0 = it[5], nspl = it[2];   // workspace slots slot0 .. slot0 + nspl - 1
  const int col = blockIdx.y, W = gridDim.y, rows = p.rows_per_wg;
  const int64_t out_row0 = int64_t(it[6]) * p.Hq + int64_t(col) * rows;
  for (int idx = blockIdx.z * blockDim.x + threadIdx.x; idx < rows * (DV / 4); idx += blockDim.x * gridDim.z) {
    const int i = idx / (DV / 4);
    const int d = 4 * (idx % (DV / 4));
    float M = -INFINITY, den = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int j0 = 0; j0 < nspl; j0 += KB) {
      float mj[KB], lj[KB];
      f32x4 vj[KB];
#pragma unroll
      for (int k = 0; k < KB; ++k) {
        const int j = min(j0 + k, nspl - 1);
        const int64_t r = (int64_t(slot0 + j) * W + col) * rows + i;
        mj[k] = j0 + k < nspl ? p.ws_stats[r * 2] : -INFINITY;
        lj[k] = p.ws_stats[r * 2 + 1];
        vj[k] = *reinterpret_cast<const f32x4*>(p.ws_o + r * DV + d);
      }
      float Mn = M;
#pragma unroll
      for (int k = 0; k < KB; ++k) Mn = fmaxf(Mn, mj[k]);
      const float sc = M == -INFINITY ? 0.f : exp2f(M - Mn);
      den *= sc;
      acc *= sc;
      M = Mn;
#pragma unroll
      for (int k = 0; k < KB; ++k) {
        const float f = mj[k] == -INFINITY ? 0.f : exp2f(mj[k] - M);
        den += f * lj[k];
        acc += f * vj[k];
      }
    }
    const float inv = 1.f / den;
    u32x2 pk;
    pk[0] = pack_bf16x2(acc[0] * inv, acc[1] * inv);
    pk[1] = pack_bf16x2(acc[2] * inv, acc[3] * inv);
    *reinterpret_cast<u32x2*>(p.out + (out_row0 + i) * DV + d) = pk;
    if (d == 0 && p.lse) p.lse[out_row0 + i] = (M + log2f(den)) * kLn2;
  }
}

// Block-table entries of one work-group's key range are staged in LDS in
// windows of kPageWin pages, so K/V gathers never wait on a dependent
// block-table load (vector loads retire in order, which would otherwise turn
// every gather into two serial memory round trips).
constexpr int kPageWin = 512;

// The running max of a row moves only when a chunk raises it by more than
// this many log2 units; in between, probabilities are taken against the
// stale max (so they stay below 2^8) and the accumulators are left alone.
constexpr float kRescaleThreshold = 8.0f;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ bool wave_any(bool pred) { return __builtin_amdgcn_ballot_w64(pred) != 0; }

// Online-softmax step of one 16-row block over one 32-key chunk.
// s[b][r]: raw score q.k of key kc0 + 16b + 4gq + r for this lane's row; with
// `masked`, keys at or past `limit` are excluded (one code path: a second
// inlined copy for the unmasked case costs registers). The scale is folded
// into the exponent: p = 2^(s * scale_log2 - m). Updates the row's max m
// (log2 units, lazily), the lane's partial sum l and the accumulators o
// (rows 4gq + r), and returns the probabilities as the bf16 A operand of P V.
template <int NACC>
__device__ __forceinline__ u32x4 softmax_chunk(const f32x4 (&s)[2], bool masked, int kc0, int limit, int gq,
                                               float scale_log2, float& m, float& l, f32x4 (&o)[NACC]) {
  float x[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = s[e >> 2][e & 3];
  if (masked) {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = kc0 + chunk_key(e, gq) < limit ? x[e] : -INFINITY;
  }
  float cmax = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
  cmax = group_max(cmax) * scale_log2;
  const bool need = cmax > m + kRescaleThreshold;
  if (wave_any(need)) {
    const float m_new = need ? cmax : m;
    const float alpha = fast_exp2(m - m_new);   // 1 if unchanged, 0 from -inf
    l *= alpha;
    m = m_new;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float ar = shfl_f(alpha, 4 * gq + r);
#pragma unroll
      for (int a = 0; a < NACC; ++a) o[a][r] *= ar;
    }
  }
  const float neg_m = m == -INFINITY ? 0.f : -m;
  u32x4 pop;
  float psum = 0.f;
#pragma unroll
  for (int e2 = 0; e2 < 4; ++e2) {
    const float p0 = fast_exp2(fmaf(x[2 * e2], scale_log2, neg_m));
    const float p1 = fast_exp2(fmaf(x[2 * e2 + 1], scale_log2, neg_m));
    psum += p0 + p1;
    pop[e2] = pack_bf16x2(p0, p1);
  }
  l += psum;
  return pop;
}

// ---------------------------------------------------------------------------
// Decode, grouped-query heads.
//
// Work-group (range r, column c) owns one balanced page range of the decode
// batch, the pieces (sequence, key range) the plan lists for it, and HW =
// rows_per_wg / G KV heads starting at c * HW. Every wave serves one of those
// heads (WPH = NW / HW waves per head, taking chunks u, u + WPH, ... of each
// piece): the work-group reads whole slot rows, so its traffic spreads over
// all memory channels instead of the subset a single head's fixed row offset
// maps to. At start it copies the block-table entries of the whole range into
// LDS; the waves then walk the range as one stream of 32-key chunks with the
// next chunk's K/V loads in flight while one is computed, across piece
// boundaries. When a wave leaves a piece it writes that piece's output (whole
// sequence) or partial (split sequence), combining through LDS first when a
// head has several waves.
//
// K reads: the A operand of S^T = K Q^T puts key n of a 16-key block in lane
// n of every lane group, so a load straight into operand layout spans 16
// keys x 64 bytes per instruction: half of each 128-byte line, which on a CU
// share streams at about 60% of the rate of whole-line reads. Each K load
// instruction instead reads 8 keys x 128 contiguous bytes (lane 8q + x: key
// q, 16-byte chunk x of one half row; at head dim 128 the two lane octets of
// a key pair take opposite halves so the LDS writes below are conflict free),
// and the chunk passes through the wave's own 32-key LDS buffer (rows
// XOR-swizzled by 16-byte chunk) on its way to the MFMA. V loads already
// cover whole rows (4 keys x 256 bytes per instruction at head dim 128).
// ---------------------------------------------------------------------------
template <int D>
struct DecodeChunk {
  static constexpr int DC = D / 32;
  using VRow = typename std::conditional<D == 128, u32x4, u32x2>::type;
  u32x4 k[2][DC];   // K of 16-key block b, load t: key 16b + kkey(t), chunk kchunk(t)
  VRow v[8];        // value dims DPL*n .. of the lane's 8 keys
};

// Bytes of one wave's K staging buffer (32 keys).
template <int D>
constexpr int decode_kstage_bytes() { return 32 * D * 2; }

// Physical 16-byte chunk of logical chunk x in key row r of a K staging
// buffer: reads of one chunk by the 16 lanes of a lane group, and the
// whole-line writes, hit 16 distinct 16-byte bank groups.
template <int D>
__device__ __forceinline__ int decode_kswz(int x, int r) {
  if constexpr (D == 128) return x ^ (r & 15);
  else return x ^ ((r >> 1) & 7);
}

// Position in a wave's chunk stream: piece i (plan item), chunk ci of it, and
// the piece's first entry in the LDS page window. Wave-uniform.
struct DecodeCursor {
  int i, ci, seq, k0, k1, poff;
};

__device__ __forceinline__ int pages_in(int k0, int k1, int P) { return (k1 - 1) / P - k0 / P + 1; }

// One decode work-group's work: balanced range `range` (-1: none) of the
// plan, column `col` of W, with threads tid = 0 .. NW*64-1, the range's
// block-table window at s_pt and NW K staging buffers at s_kst (16-byte
// aligned). Every call passes exactly one work-group barrier (two or more
// per piece with COMBINE).
template <int D, int NW, int P, bool COMBINE, bool NT>
__device__ __forceinline__ void decode_gqa_body(const AttnParams& p, int range, int col, int W, int tid,
                                                int* s_pt, uint8_t* s_kst) {
  // K/V loads marked non-temporal (read once, never reused): 7% faster on a
  // 96- or 128-CU share and 12% on the whole device than plain loads.
  constexpr int kLoadAux = NT ? 2 : 0;
  static_assert(D == 64 || D == 128, "head dim");
  constexpr int DC = D / 32;   // 32-dim chunks of the QK^T contraction
  constexpr int DPL = D / 16;  // value dims each lane owns in PV
  using Chunk = DecodeChunk<D>;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, gq = lane >> 4;
  const int G = p.G;
  const int HW = p.rows_per_wg / G;        // KV heads of this work-group
  const int WPH = max(1, NW / HW);         // waves per head
  const int hh = w / WPH, u = w % WPH;     // this wave's head within the group, rank among its waves
  const int g = col * HW + hh;             // this wave's KV head
  const bool active = hh < HW && g < p.Hkv;
  const int i_begin = range >= 0 ? p.ranges[range] : 0, i_end = range >= 0 ? p.ranges[range + 1] : 0;
  // Byte strides (the host checks that a page's slots span less than 2^31
  // bytes) and per-lane byte offsets of a chunk's loads from the page bases.
  const uint8_t* kbase_b = reinterpret_cast<const uint8_t*>(p.kc.base + int64_t(active ? g : 0) * p.kc.sh);
  const uint8_t* vbase_b = reinterpret_cast<const uint8_t*>(p.vc.base + int64_t(active ? g : 0) * p.vc.sh);
  const uint32_t ksp_b = uint32_t(p.kc.sp) * 2u, kss_b = uint32_t(p.kc.ss) * 2u;
  const uint32_t vsp_b = uint32_t(p.vc.sp) * 2u, vss_b = uint32_t(p.vc.ss) * 2u;
  const uint32_t v_lane = uint32_t(4 * gq) * vss_b + 2u * DPL * n;
  // K load t of a 16-key block: key kkey, 16-byte chunk kchunk of that key's
  // row (global byte offset k_lane[t], staging offset k_wr[t]); operand read
  // cc: key n, chunk 4cc + gq (staging offset k_rd[cc]).
  constexpr int KROW = 2 * D;
  uint8_t* const kst = s_kst + w * decode_kstage_bytes<D>();
  uint32_t k_lane[DC], k_wr[DC], k_rd[DC];
#pragma unroll
  for (int t = 0; t < DC; ++t) {
    const int q8 = lane >> 3, x8 = lane & 7;
    const int kkey = D == 128 ? 8 * (t & 1) + q8 : 8 * t + q8;
    const int kchunk = D == 128 ? 8 * ((t >> 1) ^ (q8 & 1)) + x8 : x8;
    k_lane[t] = uint32_t(kkey) * kss_b + 16u * uint32_t(kchunk);
    k_wr[t] = uint32_t(kkey * KROW + 16 * decode_kswz<D>(kchunk, kkey));
    k_rd[t] = uint32_t(n * KROW + 16 * decode_kswz<D>(4 * t + gq, n));
  }
  __shared__ float s_m[NW][16];
  __shared__ float s_l[NW][16];
  __shared__ float s_o[COMBINE ? NW : 1][16][D];   // wave combine (several waves per head)

  // The range's block-table entries, piece after piece.
  {
    int poff = 0;
    for (int i = i_begin; i < i_end; ++i) {
      const int k0 = scalar_word(p.items, 8 * i + 3), k1 = scalar_word(p.items, 8 * i + 4);
      const int32_t* bt_row = p.bt + int64_t(scalar_word(p.items, 8 * i)) * p.bt_stride + k0 / P;
      const int npg = pages_in(k0, k1, P);
      for (int t = tid; t < npg; t += NW * 64) s_pt[poff + t] = bt_row[t];
      poff += npg;
    }
  }

  // First piece at or after i (window offset poff) in which this wave has a chunk.
  auto open = [&](DecodeCursor& c, int i, int poff) {
    for (; active && i < i_end; ++i) {
      const int k0 = scalar_word(p.items, 8 * i + 3), k1 = scalar_word(p.items, 8 * i + 4);
      if (u * 32 < k1 - k0) {
        c = DecodeCursor{i, u, scalar_word(p.items, 8 * i), k0, k1, poff};
        return;
      }
      poff += pages_in(k0, k1, P);
    }
    c.i = i_end;
  };
  auto advance = [&](DecodeCursor& c) {
    c.ci += WPH;
    if (c.k0 + 32 * c.ci >= c.k1) open(c, c.i + 1, c.poff + pages_in(c.k0, c.k1, P));
  };

  // K/V loads of one chunk through buffer resources built per 16-key half
  // from scalar page bases; the record count ends at the piece's last key,
  // so loads past it read zeros and never touch memory. A cursor past the
  // end of the range still issues every load, with empty resources: the
  // same instruction stream on every path lets the compiler's wait counts
  // leave the next chunk's loads in flight (a conditional prefetch makes it
  // wait as if none had been issued).
  auto load = [&](Chunk& c, const DecodeCursor& cur) {
    const bool live = cur.i < i_end;
    const int kc0 = cur.k0 + 32 * cur.ci;
    __amdgpu_buffer_rsrc_t kr[2], vr[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int key = kc0 + 16 * b;
      // (readfirstlane keeps resources in scalar registers: one the compiler
      // sees in vector registers becomes a loop.)
      const uint32_t nvalid = uint32_t(__builtin_amdgcn_readfirstlane(live ? min(max(cur.k1 - key, 0), 16) : 0));
      const int pidx = live ? cur.poff + min(key, cur.k1 - 1) / P - cur.k0 / P : 0;
      const uint32_t pg = uint32_t(__builtin_amdgcn_readfirstlane(s_pt[pidx]));
      const uint32_t slot = uint32_t(key % P);
      kr[b] = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(kbase_b + (uint64_t(pg) * ksp_b + slot * kss_b)),
                                                0, __builtin_amdgcn_readfirstlane(int(nvalid * kss_b)), kBufferFlags);
      vr[b] = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(vbase_b + (uint64_t(pg) * vsp_b + slot * vss_b)),
                                                0, __builtin_amdgcn_readfirstlane(int(nvalid * vss_b)), kBufferFlags);
    }
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int cc = 0; cc < DC; ++cc)
        c.k[b][cc] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(kr[b], int(k_lane[cc]), 0, kLoadAux));
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int off = int(v_lane + uint32_t(e & 3) * vss_b);
      if constexpr (D == 128)
        c.v[e] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(vr[e >> 2], off, 0, kLoadAux));
      else
        c.v[e] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(vr[e >> 2], off, 0, kLoadAux));
    }
  };

  // Q as the B operand of S^T = K Q^T: column n = query head g*G + n of the
  // piece's token.
  u32x4 qop[DC];
  int q_piece = -1;
  auto load_q = [&](int i) {
    const int tok = scalar_word(p.items, 8 * i + 6);
    const bool ok = n < G;
    const uint16_t* qr = p.q + (int64_t(tok) * p.Hq + g * G + (ok ? n : 0)) * D + 8 * gq;
#pragma unroll
    for (int c = 0; c < DC; ++c) qop[c] = ok ? load16(qr + 32 * c) : zero4();
    q_piece = i;
  };

  float m = -INFINITY, l = 0.f;
  f32x4 o[DPL];
#pragma unroll
  for (int a = 0; a < DPL; ++a) o[a] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](const Chunk& c, const DecodeCursor& cur) {
    const int kc0 = cur.k0 + 32 * cur.ci;
    // K rows into the staging buffer and back in operand layout. Only this
    // wave touches its buffer and a wave's LDS accesses run in order; the
    // wave barrier keeps the compiler from moving the reads above the writes
    // (or the next chunk's writes above these reads).
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int t = 0; t < DC; ++t) *reinterpret_cast<u32x4*>(kst + k_wr[t] + 16 * KROW * b) = c.k[b][t];
    wave_lds_sync();
    f32x4 s[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      s[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int cc = 0; cc < DC; ++cc)
        s[b] = mfma_16x16x32(*reinterpret_cast<const u32x4*>(kst + k_rd[cc] + 16 * KROW * b), qop[cc], s[b]);
    }
    wave_lds_sync();
    const u32x4 pop = softmax_chunk<DPL>(s, kc0 + 32 > cur.k1, kc0, cur.k1, gq, p.scale_log2, m, l, o);
    u32x4 vop[DPL];
    if constexpr (D == 128) transpose8x8(c.v, vop);
    else transpose8x4(c.v, vop);
#pragma unroll
    for (int a = 0; a < DPL; ++a) o[a] = mfma_16x16x32(pop, vop[a], o[a]);
  };

  // Write piece i's result for this wave's head: the output of a whole
  // sequence (normalised, bf16) or the partial of a split one (fp32 numerator,
  // max and sum per row, into the piece's workspace slot); reset the state.
  // Lane (n, gq) holds rows 4gq + r of the accumulators at value dims
  // DPL*n .. DPL*n + DPL - 1.
  auto finish = [&](int i) {
    const int nspl = scalar_word(p.items, 8 * i + 2);
    const int tok = scalar_word(p.items, 8 * i + 6);
    const int64_t slot = int64_t(scalar_word(p.items, 8 * i + 7)) * W + col;   // this piece's workspace slot
    const float ltot = group_sum(l);
    if constexpr (!COMBINE) {   // one wave per head
      if (active) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = 4 * gq + r;
          const float mr = shfl_f(m, row), lr = shfl_f(ltot, row);
          if (row < G) {
            if (nspl == 1) {
              const float inv = 1.f / lr;
              uint16_t* dst = p.out + (int64_t(tok) * p.Hq + g * G + row) * D + DPL * n;
              if constexpr (DPL == 8) {
                u32x4 pk;
#pragma unroll
                for (int a = 0; a < 4; ++a) pk[a] = pack_bf16x2(o[2 * a][r] * inv, o[2 * a + 1][r] * inv);
                *reinterpret_cast<u32x4*>(dst) = pk;
              } else {
                u32x2 pk;
#pragma unroll
                for (int a = 0; a < 2; ++a) pk[a] = pack_bf16x2(o[2 * a][r] * inv, o[2 * a + 1][r] * inv);
                *reinterpret_cast<u32x2*>(dst) = pk;
              }
              if (n == 0 && p.lse) p.lse[int64_t(tok) * p.Hq + g * G + row] = (mr + log2f(lr)) * kLn2;
            } else {
              const int64_t srow = slot * p.rows_per_wg + hh * G + row;
              float* dst = p.ws_o + srow * D + DPL * n;
#pragma unroll
              for (int a4 = 0; a4 < DPL / 4; ++a4)
                *reinterpret_cast<f32x4*>(dst + 4 * a4) =
                    f32x4{o[4 * a4][r], o[4 * a4 + 1][r], o[4 * a4 + 2][r], o[4 * a4 + 3][r]};
              if (n == 0) {
                p.ws_stats[srow * 2] = mr;
                p.ws_stats[srow * 2 + 1] = lr;
              }
            }
          }
        }
      }
    } else {
      // Several waves per head: combine their states through LDS.
      lds_barrier();   // the previous piece's combine is done reading
      if (gq == 0) {
        s_m[w][n] = m;
        s_l[w][n] = ltot;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int a = 0; a < DPL; ++a) s_o[w][4 * gq + r][DPL * n + a] = o[a][r];
      lds_barrier();
      for (int idx = tid; idx < HW * G * (D / 2); idx += NW * 64) {
        const int h = idx / (G * (D / 2));
        const int row = (idx / (D / 2)) % G, d = 2 * (idx % (D / 2));
        const int gh = col * HW + h;
        if (gh >= p.Hkv) continue;
        const int w0 = h * WPH;
        float M = s_m[w0][row];
        for (int ww = 1; ww < WPH; ++ww) M = fmaxf(M, s_m[w0 + ww][row]);
        float den = 0.f, o0 = 0.f, o1 = 0.f;
        for (int ww = 0; ww < WPH; ++ww) {
          const float f = s_m[w0 + ww][row] == -INFINITY ? 0.f : fast_exp2(s_m[w0 + ww][row] - M);
          den += f * s_l[w0 + ww][row];
          o0 += f * s_o[w0 + ww][row][d];
          o1 += f * s_o[w0 + ww][row][d + 1];
        }
        if (nspl == 1) {
          const float inv = 1.f / den;
          *reinterpret_cast<uint32_t*>(p.out + (int64_t(tok) * p.Hq + gh * G + row) * D + d) =
              pack_bf16x2(o0 * inv, o1 * inv);
          if (d == 0 && p.lse) p.lse[int64_t(tok) * p.Hq + gh * G + row] = (M + log2f(den)) * kLn2;
        } else {
          const int64_t srow = slot * p.rows_per_wg + h * G + row;
          *reinterpret_cast<float2*>(p.ws_o + srow * D + d) = make_float2(o0, o1);
          if (d == 0) {
            p.ws_stats[srow * 2] = M;
            p.ws_stats[srow * 2 + 1] = den;
          }
        }
      }
    }
    m = -INFINITY;
    l = 0.f;
#pragma unroll
    for (int a = 0; a < DPL; ++a) o[a] = f32x4{0.f, 0.f, 0.f, 0.f};
  };

  // Finish every piece before i, then make sure Q is piece i's. A wave
  // finishes every piece of the range in order (several waves per head meet
  // in each combine).
  int fin = i_begin;
  auto enter = [&](int i) {
    for (; fin < i; ++fin) finish(fin);
    if (q_piece != i) load_q(i);
  };

  DecodeCursor c{i_end, 0, 0, 0, 0, 0};
  open(c, i_begin, 0);
  if (c.i < i_end) load_q(c.i);
  wait_vmem_all();
  lds_barrier();   // the page window is complete

  // Two fixed chunk buffers, the loop unrolled by two: the next chunk's loads
  // stay in flight during this chunk's math (a register copy between
  // iterations would force them to land first). Vector loads retire in
  // order, so everything a chunk's math waits for is issued before the next
  // chunk's loads: the piece change (outputs of finished pieces, Q of the
  // new one) comes first. (With the Q reload issued after them, the wait for
  // Q, merged over both paths of its branch, drained the prefetch at every
  // chunk.)
  Chunk A, B;
  load(A, c);
  while (c.i < i_end) {
    enter(c.i);
    DecodeCursor c2 = c;
    advance(c2);
    load(B, c2);
    compute(A, c);
    if (c2.i >= i_end) break;
    enter(c2.i);
    DecodeCursor c3 = c2;
    advance(c3);
    load(A, c3);
    compute(B, c2);
    c = c3;
  }
  for (; fin < i_end; ++fin) finish(fin);
}

template <int D, int NW, int P, bool COMBINE, bool NT>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2, 8)))
void decode_gqa_kernel(AttnParams p) {
  // The waves' K staging buffers, then the range's block-table entries.
  extern __shared__ __attribute__((aligned(16))) uint8_t s_dyn[];
  decode_gqa_body<D, NW, P, COMBINE, NT>(p, int(blockIdx.x), int(blockIdx.y), int(gridDim.y), int(threadIdx.x),
                                         reinterpret_cast<int*>(s_dyn + NW * decode_kstage_bytes<D>()), s_dyn);
}

// ---------------------------------------------------------------------------
// Row-parallel attention: prefill (grouped-query and latent) and latent decode.
//
// Each wave owns RB blocks of 16 query rows. The work-group streams key tiles
// of BN keys, gathered through the block table, straight from global memory
// into a ring of NS LDS stages (global_load_lds_dwordx4: lane i of a wave
// writes 16 bytes at stage + 16*i, so each instruction fills 1 KB); up to
// NS-2 tiles are in flight beyond the one being consumed, and one barrier per
// tile hands a stage over. Waits on these loads are explicit (vmcnt counts
// only them inside the loop). Row layouts:
//   kPrefillGrouped  work-group = (tile of TB*RB*16 tokens, KV head, head
//                    chunk); wave w = query head w / TB, token blocks
//                    (w % TB) * RB + rb: one K/V tile in LDS feeds every
//                    query head of the KV head.
//   kPrefillPerHead  work-group = (tile of NW*RB*16 tokens, query head).
//   kDecodeLatent    work-group = (decode item, group of NW*RB*16 heads).
//   kPrefillFlat     work-group = (tile of NW*RB*16 query rows, KV head): the
//                    rows of one KV head are (token, query head) pairs taken
//                    token-major, r = token * G + head, so every wave holds
//                    whole 16-row blocks whatever G is; wave w owns rows
//                    r0 + w*RB*16 .. +RB*16 of the tile.
// LDS rows: grouped-query K/V rows are unpadded and XOR-swizzled by 16-byte
// chunk so the MFMA operand reads are bank-conflict free; latent rows
// (576 wide) are padded by one chunk instead.
// ---------------------------------------------------------------------------
enum RowMode { kPrefillGrouped = 0, kPrefillPerHead = 1, kDecodeLatent = 2, kPrefillFlat = 3 };

typedef __attribute__((address_space(3))) uint8_t* lds_byte_ptr;

// 16-byte global -> LDS copy per lane: lane i writes lds_wave_base + 16 i
// (the LDS address goes in M0 and must be wave-uniform). Written as inline
// assembly so the compiler's wait insertion does not see an LDS write in
// flight: it would otherwise drain every outstanding tile load (vmcnt(0))
// before LDS reads it cannot prove disjoint, such as the transposing reads.
// Completion is awaited explicitly (wait_vmem) before the barrier that hands
// a stage to the readers.
__device__ __forceinline__ void dma16(const void* src, void* lds_wave_base) {
  const uint32_t m0 = uint32_t(reinterpret_cast<uintptr_t>((lds_byte_ptr)(lds_wave_base)));
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(__builtin_amdgcn_readfirstlane(m0)) : "memory");
}

// 16-byte buffer -> LDS copy per lane: lane i writes lds_wave_base + 16 i,
// reading rsrc base + voffset. The resource (page base, in SGPRs) is
// wave-uniform and the per-lane offset fixed for the launch, so a tile's
// loads cost scalar work only. Inline assembly for the same reason as dma16.
// The resource words often come straight from v_readfirstlane: a vector
// instruction writing an SGPR that a vector-memory instruction then reads
// needs 5 wait states, and the compiler's hazard check does not look inside
// inline assembly, so the block opens with them (s_nop 5: 6 wait states,
// which also covers the M0 write before an LDS DMA).
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void dma16_buf(const i32x4& rsrc, uint32_t voffset, void* lds_wave_base) {
  const uint32_t m0 = uint32_t(reinterpret_cast<uintptr_t>((lds_byte_ptr)(lds_wave_base)));
  asm volatile("s_nop 5\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voffset), "s"(rsrc),
               "{m0}"(__builtin_amdgcn_readfirstlane(m0))
               : "memory");
}

// Raw buffer resource over [base, base + bytes) from a wave-uniform address.
__device__ __forceinline__ i32x4 uniform_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{__builtin_amdgcn_readfirstlane(int32_t(uint32_t(a))),
               __builtin_amdgcn_readfirstlane(int32_t(uint32_t(a >> 32) & 0xFFFFu)),
               __builtin_amdgcn_readfirstlane(int32_t(bytes)), kBufferFlags};
}

template <int DQK, int DV, int NW, int RB, int BN, bool VALIAS, int NS>
struct RowParCfg {
  static constexpr int DC = DQK / 32;
  static constexpr int CPR = DQK / 8;                      // 16-byte chunks of a K row
  static constexpr int CPRV = VALIAS ? 0 : DV / 8;         // of a separate V row
  static constexpr int ROWB = VALIAS ? CPR + 1 : CPR;      // LDS K row stride, chunks
  static constexpr int K_SLOTS = BN * ROWB;
  static constexpr int SLOTS = K_SLOTS + BN * CPRV;
  static constexpr int TI_RAW = (SLOTS + 63) / 64;         // 1 KB loads per tile
  static constexpr int TI = (TI_RAW + NW - 1) / NW * NW;
  static constexpr int NI = TI / NW;                       // per wave per tile
  // With two stages every tile wait drains all loads, so the loads past
  // TI_RAW that only round TI up to the wave count are skipped and the stage
  // holds TI_RAW KB (this is what lets two 4-wave latent work-groups share a
  // CU's LDS). With more stages each wave counts NI loads per tile.
  static constexpr int TI_USED = NS == 2 ? TI_RAW : TI;
  static constexpr int STAGE = TI_USED * 1024;
  static constexpr int V_OFF = K_SLOTS * 16;
  static constexpr int NT = NW * 64;
  static constexpr int NACC = DV / 16;
  static constexpr size_t LDS_BYTES = size_t(NS) * STAGE + kPageWin * 4;
  static_assert(BN % 32 == 0, "key tile is a multiple of 32");
  static_assert(VALIAS || K_SLOTS % 64 == 0, "separate K and V regions start on a load boundary");
  static_assert((NS - 2) * NI < 64, "vmcnt range");
};

// Physical 16-byte chunk of logical chunk x in row r of an LDS tile.
template <int DQK, bool VALIAS>
__device__ __forceinline__ int swz_k(int x, int r) {
  if constexpr (VALIAS) return x;
  else if constexpr (DQK == 128) return x ^ (r & 15);        // 256-byte rows
  else return x ^ ((r >> 1) & 7);   // 128-byte rows; 384-byte rows (odd rows start half a bank row on)
}
template <int DV>
__device__ __forceinline__ int swz_v(int x, int r) {
  if constexpr (DV == 128) return x ^ (2 * (r & 7));
  else return x ^ (2 * ((r >> 1) & 3));
}

// vmcnt wait that leaves the loads of the last `ahead` tiles in flight
// (NI load instructions per tile per wave, at most MAXA tiles ahead).
template <int NI, int MAXA>
__device__ __forceinline__ void wait_tiles(int ahead) {
  static_assert(MAXA * NI < 64, "vmcnt range");
  if constexpr (MAXA >= 4) {
    if (ahead >= 4) { wait_vmem<4 * NI>(); return; }
  }
  if constexpr (MAXA >= 3) {
    if (ahead == 3) { wait_vmem<3 * NI>(); return; }
  }
  if constexpr (MAXA >= 2) {
    if (ahead == 2) { wait_vmem<2 * NI>(); return; }
  }
  if constexpr (MAXA >= 1) {
    if (ahead == 1) { wait_vmem<NI>(); return; }
  }
  wait_vmem<0>();
}

// Tile loads of one work-group: BN keys of K rows (and of V rows unless V
// aliases K) from the paged cache into one LDS stage, through 16-byte DMA
// loads. Load instruction j of wave w fills 1 KB of a stage: lane slot
// s = 64 * (w * NI + j) + lane is one 16-byte chunk of a K row
// (s < K_SLOTS) or of a V row. Byte offsets split into a per-lane part fixed
// for the whole launch and a per-tile part: a tile starts on a multiple of
// BN keys, so in a tile that lies below key_end the slot of row r within its
// page is r % P (pages of at most BN keys) or kb % P + r (larger pages).
// s_pt holds the block-table entries of the current page window.
template <int DQK, int DV, int NW, int BN, bool VALIAS, int NS, int P>
struct TileLoader {
  using C = RowParCfg<DQK, DV, NW, 1, BN, VALIAS, NS>;
  static_assert(VALIAS || P >= BN || (64 % C::CPR == 0 && P % (64 / C::CPR) == 0),
                "a load instruction stays in one page");
  // A whole tile whose load instructions each stay in one page (every row
  // layout but the padded latent rows with pages of at most BN keys): the
  // tile's pages are read once into scalar registers and every load goes
  // through a buffer resource on its page, with the launch-fixed per-lane
  // offsets; no per-tile vector address arithmetic.
  static constexpr bool kUniformPage = !(VALIAS && P <= BN);
  static constexpr int PPT = P <= BN ? BN / P : 1;   // pages per tile

  uint8_t* lds;
  const int* s_pt;
  int w, lane, key_end;
  const uint8_t* kbase;
  const uint8_t* vbase;
  uint32_t ksp, kss, vsp, vss;
  // Per-lane byte offsets of the loads, fixed for the launch. The two-stage
  // latent form (four waves, ten loads each per tile, two work-groups per
  // CU) forms them again at each tile instead of holding them: beside its
  // accumulators and Q they would spill.
  static constexpr bool kHoldOff = !(VALIAS && NS == 2);
  uint32_t ld_lane_off[kHoldOff ? C::NI : 1];

  __device__ __forceinline__ TileLoader(const AttnParams& p, int head_kv, uint8_t* lds_, const int* s_pt_, int w_,
                                        int lane_, int key_end_)
      : lds(lds_), s_pt(s_pt_), w(w_), lane(lane_), key_end(key_end_) {
    kbase = reinterpret_cast<const uint8_t*>(p.kc.base + int64_t(head_kv) * p.kc.sh);
    vbase = reinterpret_cast<const uint8_t*>((VALIAS ? p.kc.base : p.vc.base) +
                                             int64_t(head_kv) * (VALIAS ? p.kc.sh : p.vc.sh));
    ksp = uint32_t(p.kc.sp) * 2u;
    kss = uint32_t(p.kc.ss) * 2u;
    vsp = uint32_t(VALIAS ? p.kc.sp : p.vc.sp) * 2u;
    vss = uint32_t(VALIAS ? p.kc.ss : p.vc.ss) * 2u;
    if constexpr (kHoldOff) {
#pragma unroll
      for (int j = 0; j < C::NI; ++j) ld_lane_off[j] = form_lane_off(j, lane);
    }
  }
  __device__ __forceinline__ uint32_t form_lane_off(int j, int ln) const {
    int row;
    uint32_t xoff;
    slot_of(j, ln, row, xoff);
    return (P <= BN ? uint32_t(row % P) : uint32_t(row)) * (is_v(j) ? vss : kss) + xoff;
  }
  __device__ __forceinline__ uint32_t lane_off(int j) const {
    if constexpr (kHoldOff) {
      return ld_lane_off[j];
    } else {
      int ln = lane;
      asm volatile("" : "+v"(ln));   // keeps the arithmetic at the load, out of the loop
      return form_lane_off(j, ln);
    }
  }
  // Whether load j of this wave fills V rows (wave-uniform).
  __device__ __forceinline__ bool is_v(int j) const { return !VALIAS && (w * C::NI + j) * 64 >= C::K_SLOTS; }
  // Row and byte offset within the row of the chunk lane slot s loads.
  __device__ __forceinline__ void slot_of(int j, int ln, int& row, uint32_t& xoff) const {
    const int blk = w * C::NI + j;
    const int s = blk * 64 + ln;
    int x = 0;
    row = 0;
    if constexpr (!kHoldOff) {   // branch-free: formed again at every tile
      const int r = s / C::ROWB, pc = s - r * C::ROWB;
      const bool in = s < C::K_SLOTS;
      row = in ? r : 0;
      x = in && pc < C::CPR ? pc : 0;
    } else if (VALIAS || blk * 64 < C::K_SLOTS) {   // wave-uniform
      if (s < C::K_SLOTS) {
        row = s / C::ROWB;
        const int pc = s % C::ROWB;
        x = pc < C::CPR ? swz_k<DQK, VALIAS>(pc, row) : 0;
      }
    } else if (s < C::SLOTS) {
      const int s2 = s - C::K_SLOTS;
      row = s2 / (C::CPRV > 0 ? C::CPRV : 1);
      x = swz_v<DV>(s2 % (C::CPRV > 0 ? C::CPRV : 1), row);
    }
    xoff = 16u * uint32_t(x);
  }
  // Page of a slot within its tile (pages of at most BN keys): per lane for
  // the padded latent rows; for unpadded rows one load instruction covers
  // 64 / CPR whole rows of one page, so it is wave-uniform.
  __device__ __forceinline__ int tile_page(int j, int row) const {
    if constexpr (P > BN) return 0;
    if constexpr (VALIAS) return row / P;
    const int blk = w * C::NI + j;
    const int row0 = blk * 64 < C::K_SLOTS ? blk * 64 / C::CPR : (blk * 64 - C::K_SLOTS) / (C::CPRV > 0 ? C::CPRV : 1);
    return __builtin_amdgcn_readfirstlane(row0 / P);
  }
  __device__ __forceinline__ void issue_whole(int kb, int st, int pt_base) const {
    uint8_t* sbase = lds + st * C::STAGE;
    int pg[PPT];
#pragma unroll
    for (int t = 0; t < PPT; ++t) pg[t] = __builtin_amdgcn_readfirstlane(s_pt[kb / P - pt_base + t]);
    const uint32_t in_page = P > BN ? uint32_t(kb % P) : 0u;   // first slot of the tile in its page
#pragma unroll
    for (int j = 0; j < C::NI; ++j) {
      if constexpr (C::TI_USED < C::TI) {
        if (w * C::NI + j >= C::TI_USED) break;   // wave-uniform
      }
      const bool isv = is_v(j);
      const uint8_t* base = isv ? vbase : kbase;
      const uint32_t sp = isv ? vsp : ksp, ss = isv ? vss : kss;
      const int tp = tile_page(j, 0);
      int page = pg[0];
#pragma unroll
      for (int t = 1; t < PPT; ++t) page = tp == t ? pg[t] : page;
      const i32x4 r = uniform_rsrc(base + (uint64_t(uint32_t(page)) * sp + in_page * ss), uint32_t(min(P, BN)) * ss);
      dma16_buf(r, lane_off(j), sbase + (w * C::NI + j) * 1024);
    }
  }
  // Issue this wave's loads of the key tile starting at kb into stage st.
  // Keys past key_end read the last key's row (masked later); padding slots
  // read a dummy row.
  __device__ __forceinline__ void issue(int kb, int st, int pt_base) const {
    uint8_t* sbase = lds + st * C::STAGE;
    const bool whole = kb + BN <= key_end;
    if constexpr (kUniformPage) {
      if (whole) {
        issue_whole(kb, st, pt_base);
        return;
      }
    }
#pragma unroll
    for (int j = 0; j < C::NI; ++j) {
      if constexpr (C::TI_USED < C::TI) {
        if (w * C::NI + j >= C::TI_USED) break;   // wave-uniform
      }
      const bool isv = is_v(j);
      const uint8_t* base = isv ? vbase : kbase;
      const uint32_t sp = isv ? vsp : ksp, ss = isv ? vss : kss;
      int pidx;
      uint32_t off;
      if (whole) {
        int row = 0;
        if constexpr (VALIAS && P <= BN) {
          uint32_t xoff;
          slot_of(j, lane, row, xoff);
        }
        pidx = kb / P - pt_base + tile_page(j, row);
        off = P <= BN ? lane_off(j) : lane_off(j) + uint32_t(kb % P) * ss;
      } else {
        int row;
        uint32_t xoff;
        slot_of(j, lane, row, xoff);
        const uint32_t key = uint32_t(min(kb + row, key_end - 1));
        pidx = int(key / P) - pt_base;
        off = (key % P) * ss + xoff;
      }
      const uint32_t page = uint32_t(s_pt[pidx]);
      dma16(base + (uint64_t(page) * sp + off), sbase + (w * C::NI + j) * 1024);
    }
  }
};

// One work-group's work: item `item` of the phase, column `col`, threads
// 0 .. NW*64-1 of the work-group, the work-group's dynamic LDS.
template <int DQK, int DV, int NW, int RB, int BN, bool VALIAS, int MODE, int P, int NS, int TB>
__device__ __forceinline__ void rowpar_body(const AttnParams& p, int item, int col) {
  using C = RowParCfg<DQK, DV, NW, RB, BN, VALIAS, NS>;
  static_assert(NS >= 2 && NS <= 6, "stages");
  static_assert(BN % 32 == 0, "whole 32-key chunks per tile");
  static_assert(P % BN == 0 || BN % P == 0, "pages and tiles nest");
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];
  int* s_pt = reinterpret_cast<int*>(lds + NS * C::STAGE);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, gq = lane >> 4;
  const int32_t* it = p.items + 8 * (MODE == kDecodeLatent ? p.order[item] : item);
  const int seq = it[0];
  const int L = p.seq_lens[seq];
  const int q0 = p.qsl[seq];
  const int nq = p.qsl[seq + 1] - q0;
  const int32_t* bt_row = p.bt + int64_t(seq) * p.bt_stride;

  // Per row: query token and head, and the key limit (keys >= limit are
  // masked). Rows past the tile's end repeat its first row, so they stay
  // finite and never force masking; their results are not written.
  // wave_limit: end of the keys any row of the wave sees; wave_full: keys
  // below it are visible to every row of the wave.
  int key_begin, key_end, head_kv, wave_limit, wave_full;
  bool wave_on = true;
  int row_tok[RB], row_head[RB], row_limit[RB];
  if constexpr (MODE == kDecodeLatent) {
    key_begin = it[3];
    key_end = min(it[4], L);
    const int hg = col;
    head_kv = (hg * p.rows_per_wg) / p.G;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      row_tok[rb] = q0;
      row_head[rb] = hg * p.rows_per_wg + (w * RB + rb) * 16 + n;
      row_limit[rb] = key_end;
    }
    wave_limit = wave_full = key_end;
  } else if constexpr (MODE == kPrefillPerHead) {
    const int r0 = it[2], r1 = it[3];
    key_begin = 0;
    key_end = it[4];
    const int h = col;
    head_kv = h / p.G;
    const int wr0 = r0 + w * RB * 16;   // first row of the wave
    wave_on = wr0 < r1;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int local = wr0 + rb * 16 + n;
      const int lr = local < r1 ? local : wr0;
      row_tok[rb] = q0 + (wave_on ? lr : r0);
      row_head[rb] = h;
      row_limit[rb] = L - nq + lr + 1;
    }
    wave_limit = wave_on ? L - nq + min(r1, wr0 + RB * 16) : 0;
    wave_full = L - nq + wr0 + 1;
  } else if constexpr (MODE == kPrefillFlat) {
    const int r0 = it[2], r1 = it[3];
    key_begin = 0;
    key_end = it[4];
    head_kv = col;
    const int G = p.G;
    const int base = L - nq;                 // keys before the chunk's first token
    const int wr0 = r0 + w * RB * 16;        // first row of the wave
    wave_on = wr0 < r1;
    const int rfirst = wave_on ? wr0 : r0;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int local = rfirst + rb * 16 + n;
      const int lr = local < r1 ? local : rfirst;
      const int tok = lr / G;
      row_tok[rb] = q0 + tok;
      row_head[rb] = head_kv * G + (lr - tok * G);
      row_limit[rb] = base + tok + 1;
    }
    wave_limit = wave_on ? base + (min(r1, wr0 + RB * 16) - 1) / G + 1 : 0;
    wave_full = base + rfirst / G + 1;
  } else {
    const int r0 = it[2], r1 = it[3];
    key_begin = 0;
    key_end = it[4];
    constexpr int HPW = NW / TB;                       // query heads per work-group
    const int chunks = (p.G + HPW - 1) / HPW;
    head_kv = col / chunks;
    const int hl = (col % chunks) * HPW + w / TB;   // query head within the group
    const int wr0 = r0 + (w % TB) * RB * 16;               // first row of the wave
    wave_on = hl < p.G && wr0 < r1;
    const int h = head_kv * p.G + (hl < p.G ? hl : 0);
    const int rfirst = wr0 < r1 ? wr0 : r0;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int local = rfirst + rb * 16 + n;
      const int lr = local < r1 ? local : rfirst;
      row_tok[rb] = q0 + lr;
      row_head[rb] = h;
      row_limit[rb] = L - nq + lr + 1;
    }
    wave_limit = wave_on ? L - nq + min(r1, wr0 + RB * 16) : 0;
    wave_full = L - nq + rfirst + 1;
  }

  // Q as the B operand of S^T = K Q^T.
  u32x4 qop[RB][C::DC];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const uint16_t* qr = p.q + (int64_t(row_tok[rb]) * p.Hq + row_head[rb]) * DQK + 8 * gq;
#pragma unroll
    for (int c = 0; c < C::DC; ++c) qop[rb][c] = load16(qr + 32 * c);
  }

  float m[RB];
  // Row sums of the probabilities: through the MFMA unit against a ones
  // operand (lsum, rows 4*gq + r like the accumulators), or, for the 576-wide
  // latent rows, whose operands fill the register file, as one partial per
  // lane on the VALU (lpart, row n, this lane's keys; summed over the four
  // lane groups at the end). Both add the bf16-rounded probabilities that
  // feed the P x V product.
  constexpr bool kValuSum = VALIAS;
  f32x4 o[RB][C::NACC], lsum[RB];
  float lpart[RB];
  // Row maxima start at the lowest finite float rather than -inf: -m then
  // enters the exponent with no guard. Scores of masked keys are -inf, so a
  // row whose keys are all masked in a tile keeps this floor and adds zeros;
  // its first visible score lifts m past the rescale threshold.
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m[rb] = -FLT_MAX;
    lsum[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
    lpart[rb] = 0.f;
#pragma unroll
    for (int a = 0; a < C::NACC; ++a) o[rb][a] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const u32x4 ones = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};   // bf16 1.0 x 8

  const TileLoader<DQK, DV, NW, BN, VALIAS, NS, P> loader(p, head_kv, lds, s_pt, w, lane, key_end);
  auto issue = [&](int kb, int st, int pt_base) { loader.issue(kb, st, pt_base); };

  // Per-lane LDS byte offsets of the MFMA operand reads within a stage. The
  // row swizzles depend only on the row modulo 16 (K) or 8 (V), so they are
  // the same for every 32-key chunk and 16-key block of a tile: chunk, block
  // and stage enter as immediate offsets.
  constexpr int CH = BN / 32;                      // 32-key chunks per tile
  constexpr int KROW = C::ROWB * 16;               // LDS bytes per K row
  constexpr int VROW = VALIAS ? KROW : C::CPRV * 16;
  constexpr int NKO = VALIAS ? 1 : C::DC, NVO = VALIAS ? 1 : C::NACC;
  const int rowa0 = 4 * gq + (n >> 2);             // V row of the lane's first 4 keys
  const int cb = 8 * (n & 3);                      // byte offset of its 4 columns in a 32-byte block
  uint32_t k_off[NKO], v_off[NVO];
  if constexpr (VALIAS) {
    k_off[0] = uint32_t(n * KROW + 16 * gq);
    v_off[0] = uint32_t(rowa0 * VROW + cb);
  } else {
#pragma unroll
    for (int c = 0; c < C::DC; ++c) k_off[c] = uint32_t(n * KROW + 16 * swz_k<DQK, VALIAS>(4 * c + gq, n));
#pragma unroll
    for (int cv = 0; cv < C::NACC; ++cv) {
      const int x = 2 * cv + (cb >> 4);
      v_off[cv] = uint32_t(C::V_OFF + rowa0 * VROW + 16 * swz_v<DV>(x, rowa0) + (cb & 15));
    }
  }
  // Stage base (wave-uniform) + per-lane offset + an immediate; pointer
  // arithmetic so the constant part folds into the instruction's offset.
  auto kread = [&](const uint8_t* stage, int ch, int b, int c) {
    const uint8_t* base = stage + (VALIAS ? k_off[0] : k_off[c]);
    return *reinterpret_cast<const u32x4*>(base + ((32 * ch + 16 * b) * KROW + (VALIAS ? 64 * c : 0)));
  };
  auto vread = [&](const uint8_t* stage, int ch, int half, int cv) {
    const uint8_t* base = stage + (VALIAS ? v_off[0] : v_off[cv]);
    return lds_read_tr16(
        reinterpret_cast<const uint16_t*>(base + ((32 * ch + 16 * half) * VROW + (VALIAS ? 32 * cv : 0))));
  };

  // One key tile: S^T = K Q^T per 32-key chunk, masking (only when the tile
  // crosses a row limit), the tile max of each row, lazy rescale, then
  // probabilities and O += P V, l += P 1 per chunk. (One instance per loop:
  // a masked and an unmasked copy in one loop body would be merged by the
  // compiler at a large register cost.)
  auto compute_tile = [&](bool masked, int st, int kc0) {
    const uint8_t* stage = lds + __builtin_amdgcn_readfirstlane(st * C::STAGE);
    f32x4 s[RB][2 * CH];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < 2 * CH; ++i) s[rb][i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ch = 0; ch < CH; ++ch) {
      if constexpr (C::DC <= 4) {
        u32x4 kop[2][C::DC];
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int c = 0; c < C::DC; ++c) kop[b][c] = kread(stage, ch, b, c);
#pragma unroll
        for (int c = 0; c < C::DC; ++c)
#pragma unroll
          for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) s[rb][2 * ch + b] = mfma_16x16x32(kop[b][c], qop[rb][c], s[rb][2 * ch + b]);
      } else {
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int c = 0; c < C::DC; ++c) {
            const u32x4 kop = kread(stage, ch, b, c);
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) s[rb][2 * ch + b] = mfma_16x16x32(kop, qop[rb][c], s[rb][2 * ch + b]);
          }
      }
      // Keep each chunk's operand reads next to its products: hoisting every
      // read of the tile to the top would cost a register per value.
      __builtin_amdgcn_sched_barrier(0);
    }

    // s[rb][2ch + b][r] is the score of key kc0 + 32ch + 16b + 4gq + r for row n.
    float cmax[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      if (masked) {
#pragma unroll
        for (int i = 0; i < 2 * CH; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            s[rb][i][r] = kc0 + 16 * i + 4 * gq + r < row_limit[rb] ? s[rb][i][r] : -INFINITY;
      }
      // One chain, so that the compiler pairs it into three-input maxima.
      float mx = s[rb][0][0];
#pragma unroll
      for (int i = 0; i < 2 * CH; ++i)
#pragma unroll
        for (int r = (i == 0 ? 1 : 0); r < 4; ++r) mx = fmaxf(mx, s[rb][i][r]);
      cmax[rb] = mx;
    }
    if constexpr (RB == 2) {
      group_max2(cmax[0], cmax[1]);
    } else {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) cmax[rb] = group_max(cmax[rb]);
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) cmax[rb] *= p.scale_log2;

    // Lazy rescale: a row's max moves only when the tile max exceeds it by
    // more than the threshold; then its accumulators and sum scale by 2^(m-m').
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const bool need = cmax[rb] > m[rb] + kRescaleThreshold;
      if (wave_any(need)) {
        const float m_new = need ? cmax[rb] : m[rb];
        const float alpha = fast_exp2(m[rb] - m_new);   // 1 if unchanged, 0 from -inf
        m[rb] = m_new;
        if constexpr (kValuSum) lpart[rb] *= alpha;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float ar = shfl_f(alpha, 4 * gq + r);
          if constexpr (!kValuSum) lsum[rb][r] *= ar;
#pragma unroll
          for (int a = 0; a < C::NACC; ++a) o[rb][a][r] *= ar;
        }
      }
    }

#pragma unroll
    for (int ch = 0; ch < CH; ++ch) {
      // Probabilities 2^(s * scale_log2 - m) as the bf16 A operand of P x V.
      u32x4 pop[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const float neg_m = -m[rb];
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          const f32x4& sb = s[rb][2 * ch + (e2 >> 1)];
          const int r = 2 * (e2 & 1);
          pop[rb][e2] = pack_bf16x2(fast_exp2(fmaf(sb[r], p.scale_log2, neg_m)),
                                    fast_exp2(fmaf(sb[r + 1], p.scale_log2, neg_m)));
          if constexpr (kValuSum)
            lpart[rb] += __uint_as_float(pop[rb][e2] << 16) + __uint_as_float(pop[rb][e2] & 0xFFFF0000u);
        }
        if constexpr (!kValuSum) lsum[rb] = mfma_16x16x32(pop[rb], ones, lsum[rb]);
      }
      // Transposing LDS reads give each lane its 8 keys of value column
      // 16cv + n (keys 4gq + e and 16 + 4gq + e of the chunk).
#pragma unroll
      for (int cv = 0; cv < C::NACC; ++cv) {
        const u32x2 lo = vread(stage, ch, 0, cv);
        const u32x2 hi = vread(stage, ch, 1, cv);
        const u32x4 vop = {lo[0], lo[1], hi[0], hi[1]};
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) o[rb][cv] = mfma_16x16x32(pop[rb], vop, o[rb][cv]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Q must land before the loop: inside it vmcnt counts only the tile loads.
  wait_vmem_all();

  // Windows of kPageWin block-table entries; the tile pipeline drains at the
  // end of each window (one window covers the whole range in the usual case).
  // Iteration kt waits for tile kt, passes one barrier (every wave is done
  // with tile kt - 1, so its stage takes tile kt + NS - 1) and computes.
  // Tiles that no row of the wave masks and that still have a tile to issue
  // after them run in a loop with fixed wait counts and no masking.
  constexpr int WIN_KEYS = kPageWin * P;
  static_assert(WIN_KEYS % BN == 0, "windows hold whole tiles");
  const int last_page = key_end > 0 ? (key_end - 1) / P : 0;
  for (int wk0 = key_begin; wk0 < key_end; wk0 += WIN_KEYS) {
    const int wk1 = min(key_end, wk0 + WIN_KEYS);
    const int pt_base = wk0 / P;
    lds_barrier();
    for (int i = tid; i < kPageWin; i += C::NT) {
      const int pg = pt_base + i;
      s_pt[i] = pg <= last_page ? bt_row[pg] : 0;
    }
    wait_vmem_all();
    lds_barrier();
    const int ntiles = (wk1 - wk0 + BN - 1) / BN;
#pragma unroll
    for (int t = 0; t < NS - 1; ++t)
      if (t < ntiles) issue(wk0 + t * BN, t, pt_base);

    const int n_steady = wave_on ? max(0, min(max(0, wave_full - wk0) / BN, ntiles - (NS - 1))) : 0;
    int kt = 0;
    // (The 576-wide latent rows take every tile through the general loop:
    // a second copy of their compute would not fit two waves per SIMD.)
    for (; !VALIAS && kt < n_steady; ++kt) {
      wait_vmem<(NS - 2) * C::NI>();
      lds_barrier();
      issue(wk0 + (kt + NS - 1) * BN, (kt + NS - 1) % NS, pt_base);
      compute_tile(false, kt % NS, wk0 + kt * BN);
    }
    for (; kt < ntiles; ++kt) {
      const int kc = wk0 + kt * BN;
      wait_tiles<C::NI, NS - 2>(min(NS - 2, ntiles - 1 - kt));
      lds_barrier();
      if (kt + NS - 1 < ntiles) issue(wk0 + (kt + NS - 1) * BN, (kt + NS - 1) % NS, pt_base);
      if (!wave_on || kc >= wave_limit) continue;   // past this wave's rows: loads and barriers only
      compute_tile(kc + BN > wave_full, kt % NS, kc);
    }
  }

  // Epilogue. Lane (n, gq) holds rows 4*gq + r of each row block at value
  // columns 16*cv + n, and each row's probability sum in lsum[r] (or the
  // total of row n in ltot, from the per-lane partials).
  float ltot[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) ltot[rb] = kValuSum ? group_sum(lpart[rb]) : 0.f;
  if constexpr (MODE != kDecodeLatent) {
    if (!wave_on) return;
    const int r0 = it[2], r1 = it[3];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int blk = MODE == kPrefillGrouped ? ((w % TB) * RB + rb) : (w * RB + rb);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int local = r0 + blk * 16 + 4 * gq + r;
        const float mr = shfl_f(m[rb], 4 * gq + r);
        const float lr = kValuSum ? shfl_f(ltot[rb], 4 * gq + r) : lsum[rb][r];
        if (local < r1) {
          const float inv = 1.f / lr;
          // output row (token, query head) of this accumulator row
          int64_t orow;
          if constexpr (MODE == kPrefillFlat) {
            const int tok = local / p.G;
            orow = int64_t(q0 + tok) * p.Hq + head_kv * p.G + (local - tok * p.G);
          } else {
            orow = int64_t(q0 + local) * p.Hq + row_head[rb];
          }
          uint16_t* dst = p.out + orow * DV + n;
#pragma unroll
          for (int cv = 0; cv < C::NACC; ++cv)
            dst[16 * cv] = __builtin_bit_cast(uint16_t, (__bf16)(o[rb][cv][r] * inv));
          if (n == 0 && p.lse) p.lse[orow] = (mr + log2f(lr)) * kLn2;
        }
      }
    }
  } else {
    const int nspl = it[2];
    const int hg = col;
    const int W = gridDim.y;
    const int rows = p.rows_per_wg;
    const int64_t out_row0 = int64_t(q0) * p.Hq + int64_t(hg) * rows;
    const int64_t slot = int64_t(it[7]) * W + hg;   // this split's workspace slot
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rowi = (w * RB + rb) * 16 + 4 * gq + r;
        const float mr = shfl_f(m[rb], 4 * gq + r);
        const float lr = kValuSum ? shfl_f(ltot[rb], 4 * gq + r) : lsum[rb][r];
        if (nspl == 1) {
          const float inv = 1.f / lr;
          uint16_t* dst = p.out + (out_row0 + rowi) * DV + n;
#pragma unroll
          for (int cv = 0; cv < C::NACC; ++cv)
            dst[16 * cv] = __builtin_bit_cast(uint16_t, (__bf16)(o[rb][cv][r] * inv));
          if (n == 0 && p.lse) p.lse[out_row0 + rowi] = (mr + log2f(lr)) * kLn2;
        } else {
          float* dst = p.ws_o + (slot * rows + rowi) * DV + n;
#pragma unroll
          for (int cv = 0; cv < C::NACC; ++cv) dst[16 * cv] = o[rb][cv][r];
          if (n == 0) {
            p.ws_stats[(slot * rows + rowi) * 2] = mr;
            p.ws_stats[(slot * rows + rowi) * 2 + 1] = lr;
          }
        }
      }
    }
  }
}

template <int DQK, int DV, int NW, int RB, int BN, bool VALIAS, int MODE, int P, int NS, int TB>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(VALIAS && NS == 2 ? 2 : NW / 4)))
void rowpar_kernel(AttnParams p) {
  // Work-group -> (item, column). Decode pieces launch longest first; prefill
  // tiles are listed that way. Grouped-query prefill with a column count
  // dividing 8 runs a 1-D grid in which work-group id sits on XCD id % 8
  // (round-robin dispatch) and serves column (id % 8) % grid_y: every XCD
  // then reads the K/V of one KV head only, which its L2 can hold, instead
  // of every head's.
  int item = int(blockIdx.x), col = int(blockIdx.y);
  if ((MODE == kPrefillGrouped || MODE == kPrefillFlat) && p.xcd_remap) {
    const int x = int(blockIdx.x) & 7, j = int(blockIdx.x) >> 3;
    col = x % p.grid_y;
    item = j * (8 / p.grid_y) + x / p.grid_y;
    if (item >= p.n_items) return;
  }
  // One query head per work-group (a multiple of 8 heads): head h runs on
  // XCD h % 8 for all its tiles, tiles longest first, so each XCD's L2 holds
  // the keys and values of its own heads only.
  if (MODE == kPrefillPerHead && p.xcd_remap) {
    const int x = int(blockIdx.x) & 7, j = int(blockIdx.x) >> 3, hp8 = p.grid_y / 8;
    item = j / hp8;
    col = (j % hp8) * 8 + x;
  }
  rowpar_body<DQK, DV, NW, RB, BN, VALIAS, MODE, P, NS, TB>(p, item, col);
}

// Grouped-query prefill over flattened (token, query head) rows: WPE waves
// per SIMD are the register budget the compiler is held to, so that
// 4 * WPE / NW work-groups share a compute unit and their barriers drift
// apart. 1-D XCD-aware grid as for kPrefillGrouped.
template <int D, int NW, int RB, int BN, int P, int NS, int WPE>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(WPE)))
void flat_prefill_kernel(AttnParams p) {
  int item = int(blockIdx.x), col = int(blockIdx.y);
  if (p.xcd_remap) {
    const int x = int(blockIdx.x) & 7, j = int(blockIdx.x) >> 3;
    col = x % p.grid_y;
    item = j * (8 / p.grid_y) + x / p.grid_y;
    if (item >= p.n_items) return;
  }
  rowpar_body<D, D, NW, RB, BN, false, kPrefillFlat, P, NS, 1>(p, item, col);
}

// Per-head prefill with split-out heads (keys 192, values 128): tiles of 128
// tokens of one query head, NW waves of RB 16-row blocks, WPE waves per SIMD
// as the register budget; 1-D XCD-aware grid as in rowpar_kernel.
template <int DQK, int DV, int NW, int RB, int BN, int P, int NS, int WPE>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(WPE)))
void perhead_prefill_kernel(AttnParams p) {
  int item = int(blockIdx.x), col = int(blockIdx.y);
  if (p.xcd_remap) {
    const int x = int(blockIdx.x) & 7, j = int(blockIdx.x) >> 3, hp8 = p.grid_y / 8;
    item = j / hp8;
    col = (j % hp8) * 8 + x;
  }
  rowpar_body<DQK, DV, NW, RB, BN, false, kPrefillPerHead, P, NS, 1>(p, item, col);
}

// ---------------------------------------------------------------------------
// One-launch mixed step (grouped-query heads): work-group b takes entry
// order[b] of the plan's fused order, either one prefill work-group (tile,
// column), served by the 8-wave, 32-row-per-wave prefill body, or one
// decode work-group of RPW balanced ranges, a 4-wave decode body per range
// (RPW = 2) or one 8-wave body (RPW = 1). Prefill and decode work-groups
// share the device in the proportion the order interleaves them, instead
// of two CU-masked streams; the dispatcher hands work-groups out in id
// order as compute units free up. Decode K/V loads are non-temporal, as in
// the decode kernel. Entries < 0 are padding.
// ---------------------------------------------------------------------------
template <int D, int P, int RPW>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2)))
void fused_kernel(AttnParams pp, AttnParams pd, const int32_t* order) {
  extern __shared__ __attribute__((aligned(1024))) uint8_t lds[];
  constexpr int NS = D == 128 ? 3 : 4;
  const int e = order[blockIdx.x];
  if (e < 0) return;
  const int n_pre = pp.n_items * pp.grid_y;
  if (e < n_pre) {
    rowpar_body<D, D, 8, 2, 64, false, kPrefillGrouped, P, NS, 1>(pp, e / pp.grid_y, e % pp.grid_y);
    return;
  }
  const int j = e - n_pre;
  constexpr int DNW = 8 / RPW;
  const int sub = int(threadIdx.x) / (DNW * 64);
  const int r = RPW * j + sub;
  decode_gqa_body<D, DNW, P, false, true>(
      pd, r < pd.n_ranges ? r : -1, 0, 1, int(threadIdx.x) % (DNW * 64),
      reinterpret_cast<int*>(lds + 8 * decode_kstage_bytes<D>()) + sub * pd.range_pages,
      lds + sub * DNW * decode_kstage_bytes<D>());
}

template <int D, int P, int RPW>
static hipError_t launch_fused_t(const AttnParams& pp, const AttnParams& pd, const int32_t* order, int n_order,
                                 hipStream_t stream) {
  constexpr int NS = D == 128 ? 3 : 4;
  using C = RowParCfg<D, D, 8, 2, 64, false, NS>;
  const size_t dec_lds = 8 * size_t(decode_kstage_bytes<D>()) + size_t(RPW) * size_t(std::max(pd.range_pages, 1)) * 4;
  const size_t lds = C::LDS_BYTES > dec_lds ? C::LDS_BYTES : dec_lds;
  auto kern = fused_kernel<D, P, RPW>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(n_order), dim3(512), lds, stream, pp, pd, order);
  return hipGetLastError();
}

static hipError_t launch_merge(const AttnParams& p, int dqk, hipStream_t stream);

hipError_t launch_fused(const AttnParams& pp, const AttnParams& pd, const int32_t* order, int n_order, int dqk,
                        int ranges_per_wg, bool has_splits, hipStream_t stream) {
  if (n_order == 0) return hipSuccess;
  if (pd.P != 16 && pd.P != 64) return hipErrorInvalidValue;
  if (dqk != 64 && dqk != 128) return hipErrorInvalidValue;
  if (ranges_per_wg != 1 && ranges_per_wg != 2) return hipErrorInvalidValue;
  const bool p16 = pd.P == 16, two = ranges_per_wg == 2;
  hipError_t e;
  if (dqk == 128)
    e = p16 ? (two ? launch_fused_t<128, 16, 2>(pp, pd, order, n_order, stream)
                   : launch_fused_t<128, 16, 1>(pp, pd, order, n_order, stream))
            : (two ? launch_fused_t<128, 64, 2>(pp, pd, order, n_order, stream)
                   : launch_fused_t<128, 64, 1>(pp, pd, order, n_order, stream));
  else
    e = p16 ? (two ? launch_fused_t<64, 16, 2>(pp, pd, order, n_order, stream)
                   : launch_fused_t<64, 16, 1>(pp, pd, order, n_order, stream))
            : (two ? launch_fused_t<64, 64, 2>(pp, pd, order, n_order, stream)
                   : launch_fused_t<64, 64, 1>(pp, pd, order, n_order, stream));
  if (e != hipSuccess || !has_splits || pd.n_items == 0) return e;
  return launch_merge(pd, dqk, stream);
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

// Debug check: one work-group per sequence. The first violation found
// (kind, sequence) lands in status[0], status[1]; status must start at zero.
__global__ __launch_bounds__(256) void debug_check_kernel(const int32_t* seq_lens, const int32_t* qsl,
                                                          const int32_t* bt, int32_t bt_stride,
                                                          const int32_t* plan_lens, int32_t B, int32_t P,
                                                          int32_t num_pages, int32_t* status) {
  const int s = int(blockIdx.x);
  const int32_t L = plan_lens[s];                 // the length the plan was built for
  auto flag = [&](int kind) {
    if (atomicCAS(status, 0, kind) == 0) status[1] = s;
  };
  if (threadIdx.x == 0) {
    if (seq_lens[s] != L) flag(1);
    if (qsl[s] != plan_lens[B + s] || (s == B - 1 && qsl[B] != plan_lens[2 * B])) flag(2);
  }
  const int pages = (L + P - 1) / P;
  for (int t = int(threadIdx.x); t < pages; t += int(blockDim.x)) {
    const int32_t pg = bt[int64_t(s) * bt_stride + t];
    if (pg < 0 || pg >= num_pages) flag(3);
  }
}

// Per-device status words of the debug check, resolved once per device.
static __device__ int32_t debug_status[2];
static std::mutex g_debug_mu;
static int32_t* g_debug_ptr[64] = {};

hipError_t debug_check(const int32_t* seq_lens, const int32_t* qsl, const int32_t* bt, int32_t bt_stride,
                       const int32_t* plan_lens, int32_t num_seqs, int32_t P, int32_t num_pages, int32_t* kind,
                       int32_t* seq, hipStream_t stream) {
  *kind = 0;
  *seq = -1;
  if (num_seqs == 0) return hipSuccess;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  int32_t* status = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_debug_mu);
    if (!g_debug_ptr[dev]) {
      void* ptr = nullptr;
      if ((e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(debug_status))) != hipSuccess) return e;
      g_debug_ptr[dev] = static_cast<int32_t*>(ptr);
    }
    status = g_debug_ptr[dev];
  }
  if ((e = launch_fill_zero(status, 8, stream)) != hipSuccess) return e;
  hipLaunchKernelGGL(debug_check_kernel, dim3(num_seqs), dim3(256), 0, stream, seq_lens, qsl, bt, bt_stride,
                     plan_lens, num_seqs, P, num_pages, status);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  int32_t h[2] = {0, -1};
  if ((e = hipMemcpyAsync(h, status, sizeof(h), hipMemcpyDeviceToHost, stream)) != hipSuccess) return e;
  if ((e = hipStreamSynchronize(stream)) != hipSuccess) return e;
  *kind = h[0];
  *seq = h[1];
  return hipSuccess;
}

__global__ void fill_zero_kernel(uint32_t* p, size_t words) {
  for (size_t i = blockIdx.x * size_t(blockDim.x) + threadIdx.x; i < words; i += size_t(gridDim.x) * blockDim.x)
    p[i] = 0u;
}

// ---------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------
// Allow a kernel the dynamic LDS it launches with. The attribute is set on
// every launch (it is a cheap host-side call), so it holds on whichever device
// is current and a transient failure is not remembered.
static hipError_t set_dynamic_lds(const void* kern, size_t bytes) {
  return hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, int(bytes));
}

template <int DQK, int DV, int NW, int RB, int BN, bool VALIAS, int MODE, int P, int NS, int TB = 1>
static hipError_t launch_rowpar(const AttnParams& p, dim3 grid, hipStream_t stream) {
  using C = RowParCfg<DQK, DV, NW, RB, BN, VALIAS, NS>;
  auto kern = rowpar_kernel<DQK, DV, NW, RB, BN, VALIAS, MODE, P, NS, TB>;
  const hipError_t attr = set_dynamic_lds(reinterpret_cast<const void*>(kern), C::LDS_BYTES);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kern, grid, dim3(C::NT), C::LDS_BYTES, stream, p);
  return hipGetLastError();
}

template <int D, int P>
static hipError_t launch_decode_gqa(const AttnParams& p, hipStream_t stream) {
  // One work-group per (balanced range, KV head); the waves' K staging
  // buffers and the range's block-table entries take dynamic LDS.
  // Four waves when the work-group serves at most four KV heads, else eight
  // (one per head).
  const dim3 grid(p.n_ranges, p.grid_y);
  const size_t window = size_t(std::max(p.range_pages, 1)) * 4;   // a dead cursor reads entry 0
  const int hw = p.rows_per_wg / p.G;
  auto go = [&](auto kern, int nw) {
    const size_t lds = size_t(nw) * decode_kstage_bytes<D>() + window;
    const hipError_t attr = set_dynamic_lds(reinterpret_cast<const void*>(kern), lds);
    if (attr != hipSuccess) return attr;
    hipLaunchKernelGGL(kern, grid, dim3(nw * 64), lds, stream, p);
    return hipGetLastError();
  };
  if (hw <= 2) return go(decode_gqa_kernel<D, 4, P, true, true>, 4);   // several waves per head, combined through LDS
  if (hw <= 4) return go(decode_gqa_kernel<D, 4, P, false, true>, 4);
  return go(decode_gqa_kernel<D, 8, P, false, true>, 8);
}

static hipError_t launch_decode_kernel(const AttnParams& p, int dqk, hipStream_t stream) {
  const bool p16 = p.P == 16;
  if (p.P != 16 && p.P != 64) return hipErrorInvalidValue;
  const dim3 pieces(p.n_items, p.grid_y);
  switch (dqk) {
    case 128: return p16 ? launch_decode_gqa<128, 16>(p, stream) : launch_decode_gqa<128, 64>(p, stream);
    case 64: return p16 ? launch_decode_gqa<64, 16>(p, stream) : launch_decode_gqa<64, 64>(p, stream);
    case 576:   // one work-group per (piece, group of 128 or 64 heads), a wave per 16 heads;
                // 64-head groups take two LDS stages so that two work-groups share a CU
      if (p.rows_per_wg == 128)
        return p16 ? launch_rowpar<576, 512, 8, 1, 32, true, kDecodeLatent, 16, 3>(p, pieces, stream)
                   : launch_rowpar<576, 512, 8, 1, 32, true, kDecodeLatent, 64, 3>(p, pieces, stream);
      return p16 ? launch_rowpar<576, 512, 4, 1, 32, true, kDecodeLatent, 16, 2>(p, pieces, stream)
                 : launch_rowpar<576, 512, 4, 1, 32, true, kDecodeLatent, 64, 2>(p, pieces, stream);
    default: return hipErrorInvalidValue;
  }
}

// Merge: one work-group per (split sequence, column, slice of the output
// rows), each thread at most a few (row, 4 columns) outputs so all their
// loads are in flight together.
static hipError_t launch_merge(const AttnParams& p, int dqk, hipStream_t stream) {
  if (p.n_merge == 0) return hipSuccess;
  const int dv = dqk == 576 ? 512 : dqk;
  const int units = p.rows_per_wg * (dv / 4);
  const dim3 mgrid(p.n_merge, p.grid_y, std::min(8, (units + 255) / 256));
  switch (dqk) {
    case 128: hipLaunchKernelGGL(merge_kernel<128>, mgrid, dim3(256), 0, stream, p); break;
    case 64: hipLaunchKernelGGL(merge_kernel<64>, mgrid, dim3(256), 0, stream, p); break;
    case 576: hipLaunchKernelGGL(merge_kernel<512>, mgrid, dim3(256), 0, stream, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_decode_merge(const AttnParams& p, int dqk, hipStream_t stream) { return launch_merge(p, dqk, stream); }

hipError_t launch_decode(const AttnParams& p, int dqk, bool has_splits, hipStream_t stream) {
  if (p.n_items == 0) return hipSuccess;
  hipError_t e = launch_decode_kernel(p, dqk, stream);
  if (e != hipSuccess || !has_splits) return e;
  return launch_merge(p, dqk, stream);
}

// Grouped-query prefill: one wave per query head of a KV head (4 waves when
// the group has at most 4 heads, else 8), bm/16 token blocks per wave. The
// 16-wave form takes 64-key tiles (one work-group per CU); the smaller forms
// take 32-key tiles in three stages (50 KB of LDS at d = 128), so that two or
// more work-groups share a CU and their barriers do not line up.
template <int D, int P>
static hipError_t launch_prefill_grouped(const AttnParams& p, int bm, dim3 grid, hipStream_t stream) {
  constexpr int BN = 64;
  constexpr int NS = D == 128 ? 3 : 4;
  const bool narrow = p.G <= 4;
  if (bm == 32)
    return narrow ? launch_rowpar<D, D, 8, 1, 32, false, kPrefillGrouped, P, 3, 2>(p, grid, stream)
                  : launch_rowpar<D, D, 16, 1, BN, false, kPrefillGrouped, P, NS, 2>(p, grid, stream);
  if (bm == 16)
    return narrow ? launch_rowpar<D, D, 4, 1, 32, false, kPrefillGrouped, P, 3>(p, grid, stream)
                  : launch_rowpar<D, D, 8, 1, 32, false, kPrefillGrouped, P, 3>(p, grid, stream);
  return hipErrorInvalidValue;
}

template <int DQK, int DV, int NW, int RB, int BN, int P, int NS, int WPE>
static hipError_t launch_perhead_t(const AttnParams& p, dim3 grid, hipStream_t stream) {
  using C = RowParCfg<DQK, DV, NW, RB, BN, false, NS>;
  auto kern = perhead_prefill_kernel<DQK, DV, NW, RB, BN, P, NS, WPE>;
  const hipError_t attr = set_dynamic_lds(reinterpret_cast<const void*>(kern), C::LDS_BYTES);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kern, grid, dim3(C::NT), C::LDS_BYTES, stream, p);
  return hipGetLastError();
}

template <int D, int NW, int RB, int BN, int P, int NS, int WPE>
static hipError_t launch_flat_t(const AttnParams& p, dim3 grid, hipStream_t stream) {
  using C = RowParCfg<D, D, NW, RB, BN, false, NS>;
  auto kern = flat_prefill_kernel<D, NW, RB, BN, P, NS, WPE>;
  const hipError_t attr = set_dynamic_lds(reinterpret_cast<const void*>(kern), C::LDS_BYTES);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kern, grid, dim3(C::NT), C::LDS_BYTES, stream, p);
  return hipGetLastError();
}

// Flattened-row prefill: tiles of 128 (token, query head) rows, four waves
// of 32 rows (two 16-row blocks each, so every K/V operand read from LDS
// feeds two products), 32-key tiles in three stages (50 KB of LDS at head
// dim 128) and at most 168 registers, so that three work-groups share a
// compute unit and their barriers drift apart.
template <int D, int P>
static hipError_t launch_prefill_flat(const AttnParams& p, int bm, dim3 grid, hipStream_t stream) {
  if (bm == 128) return launch_flat_t<D, 4, 2, 32, P, 3, 3>(p, grid, stream);
  return hipErrorInvalidValue;
}

template <int P>
static hipError_t launch_prefill_p(const AttnParams& p, int dqk, int bm, dim3 grid, hipStream_t stream) {
  if ((dqk == 128 || dqk == 64) && bm >= 64) {
    AttnParams q = p;
    if (8 % p.grid_y == 0) {
      q.xcd_remap = 1;
      grid = dim3((p.n_items * p.grid_y + 7) / 8 * 8, 1);
    }
    return dqk == 128 ? launch_prefill_flat<128, P>(q, bm, grid, stream) : launch_prefill_flat<64, P>(q, bm, grid, stream);
  }
  if (dqk == 128 || dqk == 64) {
    // XCD-aware 1-D grid when the column count divides 8 (see rowpar_kernel).
    AttnParams q = p;
    if (8 % p.grid_y == 0) {
      q.xcd_remap = 1;
      grid = dim3((p.n_items * p.grid_y + 7) / 8 * 8, 1);
    }
    return dqk == 128 ? launch_prefill_grouped<128, P>(q, bm, grid, stream)
                      : launch_prefill_grouped<64, P>(q, bm, grid, stream);
  }
  // One work-group per (tile, query head), a wave per 16 rows (32 with the
  // heads split out); XCD-aware 1-D grid when the head count is a multiple
  // of 8. Latent 64-row tiles run
  // four waves over two LDS stages, so that two work-groups share a CU
  // (with three stages one work-group of four waves held the CU alone: 1.8x
  // slower).
  if (p.grid_y % 8 == 0) {
    AttnParams q = p;
    q.xcd_remap = 1;
    const dim3 g1(p.n_items * p.grid_y, 1);
    if (dqk == 576 && bm == 128) return launch_rowpar<576, 512, 8, 1, 32, true, kPrefillPerHead, P, 3>(q, g1, stream);
    if (dqk == 576 && bm == 64) return launch_rowpar<576, 512, 4, 1, 32, true, kPrefillPerHead, P, 2>(q, g1, stream);
    if constexpr (P == 64) {
      if (dqk == 192 && bm == 128) return launch_perhead_t<192, 128, 4, 2, 32, 64, 3, 2>(q, g1, stream);
    }
    return hipErrorInvalidValue;
  }
  if (dqk == 576 && bm == 128) return launch_rowpar<576, 512, 8, 1, 32, true, kPrefillPerHead, P, 3>(p, grid, stream);
  if (dqk == 576 && bm == 64) return launch_rowpar<576, 512, 4, 1, 32, true, kPrefillPerHead, P, 2>(p, grid, stream);
  // Heads split out (keys 192, values 128): one work-group per (128-token
  // tile, query head), four waves of 32 rows (two 16-row blocks each, so
  // every K/V operand read from LDS feeds two products); 32-key tiles in
  // three stages (62 KB of LDS) at 205 VGPRs, so two work-groups share a CU.
  // (Eight waves of 16 rows, 122 VGPRs: 820 against 774 us on the
  // 4096-token prompt; a 168-register budget for three per CU spills.)
  if constexpr (P == 64) {
    if (dqk == 192 && bm == 128) return launch_perhead_t<192, 128, 4, 2, 32, 64, 3, 2>(p, grid, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_prefill(const AttnParams& p, int dqk, int bm, hipStream_t stream) {
  if (p.n_items == 0) return hipSuccess;
  const dim3 grid(p.n_items, p.grid_y);
  if (p.P == 16) return launch_prefill_p<16>(p, dqk, bm, grid, stream);
  if (p.P == 64) return launch_prefill_p<64>(p, dqk, bm, grid, stream);
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
