// Host planner: validation, phase classification, decode split-K partition,
// prefill tile list and the co-run CU split. Pure integer (and one cost-model
// comparison in double) host code; it makes no HIP call, so it runs and is
// tested without a GPU.
//
// The paper's daemon validates each request and places it in a per-phase
// queue before dispatch (Sec. 3.2; Sec. 3.4 "Phase-Aware Dispatch"). For one
// mixed batch that becomes: classify each sequence by its number of new tokens
// (one -> decode, two or more -> prefill, none -> nothing), then lay out each
// phase's work so one kernel launch per phase covers the batch.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>

#include "host_common.h"

namespace flexattn {

namespace {

thread_local std::string g_last_error;

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool supported_dims(const flex_attn_shape& s) {
  const int dq = s.head_dim_qk, dv = s.head_dim_v;
  const bool gqa = (dq == 64 && dv == 64) || (dq == 128 && dv == 128);
  const bool latent = dq == 576 && dv == 512;
  const bool split = dq == 192 && dv == 128;   // latent attention with heads split out (prefill)
  if (!gqa && !latent && !split) return false;
  if (s.page_size != 16 && s.page_size != 64) return false;
  if (latent) return s.v_aliases_k && s.num_q_heads % kLatentRowsPerWG == 0;
  if (split) return !s.v_aliases_k && s.page_size == 64 && s.num_q_heads / s.num_kv_heads <= 16;
  return s.num_q_heads / s.num_kv_heads <= 16;
}

}  // namespace

// FLEX_ATTN_LOG=1: one summary line per plan on stderr; 2: also every work
// item.
int log_level() {
  static const int level = [] {
    const char* v = std::getenv("FLEX_ATTN_LOG");
    return v ? std::atoi(v) : 0;
  }();
  return level;
}

void log_plan(const ::flex_attn_plan_t& p) {
  const flex_attn_plan_info& i = p.info;
  std::fprintf(stderr,
               "flexattn plan: %d seqs (%d decode, %d prefill); decode %d pieces in %d ranges x %d columns, "
               "%d split seqs, %d pages/range; prefill %d tiles x %d (bm %d); CUs decode %d / prefill %d; "
               "%d words, workspace %zu B, fused %d\n",
               i.num_seqs, i.n_decode_seqs, i.n_prefill_seqs, i.n_decode_items, i.n_decode_ranges,
               i.decode_wg_width, i.n_split_seqs, i.pages_per_split, i.n_prefill_items, i.prefill_grid_y, i.bm,
               i.cus_decode, i.cus_prefill, i.plan_words, i.workspace_bytes, i.n_fused_wgs);
  if (log_level() < 2) return;
  const int32_t* w = p.words.data();
  for (int32_t k = 0; k < i.n_decode_items; ++k) {
    const int32_t* it = w + w[H_OFF_DEC] + kItemWords * k;
    std::fprintf(stderr, "  decode %d: seq %d piece %d/%d keys [%d, %d) slot %d\n", k, it[0], it[1], it[2], it[3],
                 it[4], it[7]);
  }
  for (int32_t k = 0; k < i.n_prefill_items; ++k) {
    const int32_t* it = w + w[H_OFF_PRE] + kItemWords * k;
    std::fprintf(stderr, "  prefill %d: seq %d tile %d rows [%d, %d) key_end %d\n", k, it[0], it[1], it[2], it[3],
                 it[4]);
  }
}

int check_shape(const flex_attn_shape& sh) {
  if (sh.num_q_heads <= 0 || sh.num_kv_heads <= 0 || sh.num_q_heads % sh.num_kv_heads)
    return set_error(FLEX_ERR_INVALID_ARG, "num_q_heads must be a positive multiple of num_kv_heads");
  if (!std::isfinite(sh.sm_scale) || !(sh.sm_scale > 0.0f))
    return set_error(FLEX_ERR_INVALID_ARG, "sm_scale must be finite and positive");
  if (sh.v_aliases_k && (sh.num_kv_heads != 1 || sh.head_dim_v > sh.head_dim_qk))
    return set_error(FLEX_ERR_INVALID_ARG, "v_aliases_k needs one KV head and head_dim_v <= head_dim_qk");
  if (!supported_dims(sh))
    return set_error(FLEX_ERR_UNSUPPORTED, "shape outside (64,64)/(128,128) GQA with group <= 16, "
                                           "(576,512) aliased latent with Hq % 64 == 0, page 16/64, "
                                           "or (192,128) with group <= 16, page 64");
  return FLEX_OK;
}

int set_error(int status, const std::string& msg) {
  g_last_error = msg;
  return status;
}

void clear_error() { g_last_error.clear(); }

const char* last_error() { return g_last_error.c_str(); }

}  // namespace flexattn

using namespace flexattn;

extern "C" const char* flex_attn_status_string(int status) {
  switch (status) {
    case FLEX_OK: return "ok";
    case FLEX_ERR_INVALID_ARG: return "invalid argument";
    case FLEX_ERR_UNSUPPORTED: return "unsupported shape or option";
    case FLEX_ERR_WORKSPACE: return "buffer too small";
    case FLEX_ERR_HIP: return "HIP runtime error";
    case FLEX_ERR_INTERNAL: return "internal error";
    default: return "unknown status";
  }
}

extern "C" const char* flex_attn_last_error(void) { return flexattn::last_error(); }

extern "C" int flex_attn_plan(const flex_attn_shape* shape, const flex_attn_plan_opts* opts,
                              int32_t num_seqs, const int32_t* qsl, const int32_t* seq_lens,
                              int32_t max_pages_per_seq, flex_attn_plan_t** out_plan) {
  clear_error();
  if (!out_plan) return set_error(FLEX_ERR_INVALID_ARG, "out_plan is NULL");
  *out_plan = nullptr;
  if (!shape) return set_error(FLEX_ERR_INVALID_ARG, "shape is NULL");
  if (num_seqs < 0) return set_error(FLEX_ERR_INVALID_ARG, "num_seqs < 0");
  if (!qsl || (num_seqs > 0 && !seq_lens))
    return set_error(FLEX_ERR_INVALID_ARG, "query_start_loc or seq_lens is NULL");
  const flex_attn_shape sh = *shape;
  if (const int st = check_shape(sh); st != FLEX_OK) return st;

  flex_attn_plan_opts o;
  std::memset(&o, 0, sizeof(o));
  if (opts) o = *opts;
  const bool latent = sh.head_dim_qk == 576;
  // (192, 128): latent attention with its heads split out (keys 128 + 64
  // rope, values 128 per head), the layout in which a long prompt costs the
  // fewest flops. Prefill only: every sequence with new tokens, one token
  // included, runs as a prefill tile of one query head.
  const bool split = sh.head_dim_qk == 192;
  const int64_t cus_total = o.cus_total ? o.cus_total : 256;
  // Grouped-query decode: one work-group per CU walking a long range measured
  // fastest; latent decode launches one work-group per piece, so more pieces.
  const int64_t wg_per_cu = o.wg_per_cu ? o.wg_per_cu : (sh.head_dim_qk == 576 ? 2 : 1);
  const int64_t min_tokens = o.min_split_tokens ? o.min_split_tokens : 256;
  const int64_t granule = o.split_granule ? o.split_granule : 32;
  int32_t bm = o.bm ? o.bm : (latent || split ? 128 : 0);   // grouped-query default: chosen below
  if (cus_total < 1 || wg_per_cu < 1 || min_tokens < 1 || granule < 1)
    return set_error(FLEX_ERR_INVALID_ARG, "plan options must be positive");
  if (o.decode_tail < -1 || o.decode_tail > 0) return set_error(FLEX_ERR_INVALID_ARG, "decode_tail must be 0 or -1");
  if (o.cus_decode < -1 || o.cus_decode > cus_total)
    return set_error(FLEX_ERR_INVALID_ARG, "cus_decode must be -1, 0 or in [1, cus_total]");
  if (latent ? (bm != 64 && bm != 128) : split ? bm != 128 : (bm != 0 && bm != 16 && bm != 32 && bm != 128))
    return set_error(FLEX_ERR_UNSUPPORTED,
                     "bm must be 16, 32 or 128 (grouped-query), 64 or 128 (latent layout), 128 (192/128 layout)");
  if (max_pages_per_seq < 0) return set_error(FLEX_ERR_INVALID_ARG, "max_pages_per_seq < 0");
  if (num_seqs > 0 && qsl[0] != 0) return set_error(FLEX_ERR_INVALID_ARG, "query_start_loc[0] != 0");

  const int64_t P = sh.page_size;
  for (int32_t s = 0; s < num_seqs; ++s) {
    const int64_t n = int64_t(qsl[s + 1]) - qsl[s];
    const int64_t L = seq_lens[s];
    if (n < 0) return set_error(FLEX_ERR_INVALID_ARG, "query_start_loc decreases at " + std::to_string(s));
    if (L < 0 || n > L)
      return set_error(FLEX_ERR_INVALID_ARG, "sequence " + std::to_string(s) + ": need 0 <= n <= L");
    if (L > int64_t(max_pages_per_seq) * P)
      return set_error(FLEX_ERR_INVALID_ARG, "sequence " + std::to_string(s) + ": L > max_pages_per_seq * page_size");
  }

  // Decode work-groups per key range: one per group of up to 8 KV heads for
  // grouped-query attention (a work-group then reads whole slot rows, which
  // spreads its stream over every memory channel); for the latent layout one
  // per 128 query heads (eight waves of 16 heads share each key tile), or per
  // 64 when 128 does not divide Hq.
  const int32_t heads_per_wg = std::min(sh.num_kv_heads, kDecodeHeadsPerWG);
  const int32_t latent_rows = sh.num_q_heads % kLatentRowsPerWGWide == 0 ? kLatentRowsPerWGWide : kLatentRowsPerWG;
  const int32_t W = latent ? sh.num_q_heads / latent_rows : int32_t(cdiv(sh.num_kv_heads, heads_per_wg));
  // Prefill work-groups per tile: one per query head (latent layout), or one per
  // KV head and group of up to 8 of its query heads (grouped-query layout).
  const int32_t G = sh.num_q_heads / sh.num_kv_heads;

  const int32_t rows_per_wg = latent ? latent_rows : heads_per_wg * (sh.num_q_heads / sh.num_kv_heads);
  std::vector<int32_t> dec, pre;
  for (int32_t s = 0; s < num_seqs; ++s) {
    const int32_t n = qsl[s + 1] - qsl[s];
    if (n == 1 && !split) dec.push_back(s);
    else if (n >= 1) pre.push_back(s);
  }

  // Algorithmic work of each phase (feeds the cost model and the plan info).
  const int64_t kv_row = int64_t(sh.num_kv_heads) * 2 *
                         (sh.v_aliases_k ? sh.head_dim_qk : sh.head_dim_qk + sh.head_dim_v);
  int64_t dec_bytes = 0;
  for (int32_t s : dec) dec_bytes += int64_t(seq_lens[s]) * kv_row;
  int64_t pre_flops = 0;
  for (int32_t s : pre) {
    const int64_t n = qsl[s + 1] - qsl[s], L = seq_lens[s];
    pre_flops += int64_t(sh.num_q_heads) * 2 * (sh.head_dim_qk + sh.head_dim_v) *
                 (n * (L - n) + n * (n + 1) / 2);
  }

  // Grouped-query prefill tiles: 128 flattened rows (a row is a (token,
  // query head) pair of one KV head, token-major: every 16-row block of a
  // wave is full whatever the group size) when the batch gives every
  // prefill CU at least four such work-groups, or, on a co-run share, when
  // they all fit in one round (three flat work-groups are resident per CU);
  // else 32 tokens, whose larger work-groups fill a CU one at a time and
  // leave no short last round. (On the whole device the one-round case runs
  // alike either way, and 32-token tiles keep the one-launch order.)
  int64_t flat_wgs = 0;
  for (int32_t s : pre) flat_wgs += cdiv(int64_t(qsl[s + 1] - qsl[s]) * G, 128) * sh.num_kv_heads;
  auto default_bm = [&](int64_t cus) -> int32_t {
    const bool share = cus < cus_total;
    return flat_wgs >= 4 * cus || (share && flat_wgs <= kFlatResidentPerCu * cus) ? 128 : 32;
  };
  // Cost-model prefill time on `cus` CUs (seconds). Grouped-query shapes:
  // the work at the per-CU rate or the largest work-group's (every key of
  // its sequence) at one work-group's rate, whichever is longer, plus the
  // launch latency; other layouts: the work at the per-CU rate.
  const int32_t bm_opt = bm;
  auto prefill_time = [&](int64_t cus, double fl_cu) -> double {
    const double t_work = double(pre_flops) / (double(cus) * fl_cu);
    if (latent || split) return t_work;
    const int32_t b = bm_opt ? bm_opt : default_bm(cus);
    double tile = 0.0;
    for (int32_t s : pre) {
      const int64_t n = qsl[s + 1] - qsl[s];
      const int64_t rows = b == 128 ? std::min<int64_t>(128, n * G) : std::min<int64_t>(b, n) * std::min(G, 8);
      tile = std::max(tile, double(rows) * double(seq_lens[s]) * double(2 * (sh.head_dim_qk + sh.head_dim_v)));
    }
    const double share = b == 128 ? kFlatWgCuShare : 1.0;
    return std::max(t_work, tile / (share * fl_cu)) + kPrefillLaunchSec;
  };

  // Co-run CU split: explicit, or the cost model's argmin of the step time:
  // the slower phase, or with a decode tail (grouped-query plans) the
  // prefill plus what decode has left by then at the device's streaming rate.
  int64_t cus_decode;
  if (o.cus_decode == 0 || dec.empty() || pre.empty()) {
    cus_decode = cus_total;
  } else if (o.cus_decode > 0) {
    cus_decode = o.cus_decode;
  } else {
    const double hbm = (o.hbm_gbps != 0.0 ? o.hbm_gbps : kDefaultHbmGBps) * 1e9;
    const double bw_cu = (o.decode_gbps_per_cu != 0.0 ? o.decode_gbps_per_cu : kDefaultDecodeGBpsPerCU) * 1e9;
    const double fl_cu = (o.prefill_tflops_per_cu != 0.0 ? o.prefill_tflops_per_cu : kDefaultPrefillTFlopsPerCU) * 1e12;
    const bool tail_model = !latent && !split && o.decode_tail == 0;
    const double r_all = std::min(hbm, double(cus_total) * bw_cu);
    int64_t best = -1;
    double best_t = 0.0;
    for (int64_t nd = granule; nd < cus_total; nd += granule) {
      const double r_share = std::min(hbm, double(nd) * bw_cu);
      const double t_dec = double(dec_bytes) / r_share;
      const double t_pre = prefill_time(cus_total - nd, fl_cu);
      double t = std::max(t_dec, t_pre);
      if (tail_model) {
        const double rest = double(dec_bytes) - r_share * t_pre;
        t = rest > 0.0 ? t_pre + rest / r_all : t_pre;
      }
      if (best < 0 || t < best_t) { best = nd; best_t = t; }
    }
    cus_decode = best > 0 ? best : cus_total;
  }
  const int64_t cus_prefill =
      (!dec.empty() && !pre.empty() && cus_decode < cus_total) ? cus_total - cus_decode : cus_total;

  if (bm == 0) bm = default_bm(cus_prefill);   // grouped-query tile height (rule above)
  const bool flat = !latent && !split && bm == 128;
  const int32_t pre_grid_y =
      latent || split ? sh.num_q_heads : flat ? sh.num_kv_heads : sh.num_kv_heads * ((G + 7) / 8);

  // Decode partition (balanced split-K): the pages of all decode sequences,
  // concatenated in batch order, are cut into near-equal ranges, one
  // work-group column each, aiming at wg_per_cu resident work-groups per
  // decode CU. A piece is the overlap of a range with one sequence; pieces
  // are listed by range (batch order, keys ascending) and the list index is
  // the piece's workspace slot, so a sequence's pieces are consecutive.
  //
  // Decode tail (grouped-query co-run plans): the decode share streams pages
  // [0, TA) while the prefill runs; pages [TA, T) form a second group of
  // ranges, sized for the prefill share, that runs on the prefill stream
  // once the prefill is done (both groups then stream together until both
  // end). TA follows the cost model: what the decode share covers during the
  // prefill, plus its share of the rest at the device's streaming rate.
  const int64_t min_pps = cdiv(min_tokens, P);
  std::vector<int64_t> start(dec.size() + 1, 0);   // first global page of each decode sequence
  for (size_t d = 0; d < dec.size(); ++d) start[d + 1] = start[d] + cdiv(seq_lens[dec[d]], P);
  const int64_t T = start[dec.size()];
  int64_t TA = T;
  if (!latent && !split && o.decode_tail == 0 && cus_prefill < cus_total && T > 1) {
    const double hbm = (o.hbm_gbps != 0.0 ? o.hbm_gbps : kDefaultHbmGBps) * 1e9;
    const double bw_cu = (o.decode_gbps_per_cu != 0.0 ? o.decode_gbps_per_cu : kDefaultDecodeGBpsPerCU) * 1e9;
    const double fl_cu = (o.prefill_tflops_per_cu != 0.0 ? o.prefill_tflops_per_cu : kDefaultPrefillTFlopsPerCU) * 1e12;
    const double r_share = std::min(hbm, double(cus_decode) * bw_cu);   // decode beside the prefill
    const double r_all = std::min(hbm, double(cus_total) * bw_cu);      // after it
    const double t_pre = prefill_time(cus_prefill, fl_cu);
    const double during = r_share * t_pre;
    if (during < double(dec_bytes)) {
      const double t_rest = (double(dec_bytes) - during) / r_all;
      const double share_rest = r_all * (double(cus_decode) / double(cus_total)) * t_rest;
      const double frac = (during + share_rest) / double(dec_bytes);
      TA = std::min(T - 1, std::max(int64_t(1), int64_t(std::floor(frac * double(T)))));
    }
  }
  const int64_t TB = T - TA;
  // Ranges per group (at least ceil(pages / kMaxRangePages): a range's
  // block-table entries are staged in LDS).
  auto n_ranges = [&](int64_t pages, int64_t cus) -> int64_t {
    if (pages == 0) return 0;
    return std::max<int64_t>({int64_t(1), std::min<int64_t>(cus * wg_per_cu / W, pages / min_pps),
                              cdiv(pages, kMaxRangePages)});
  };
  const int64_t RA = dec.empty() ? 0 : n_ranges(TA, cus_decode);
  const int64_t RB = dec.empty() ? 0 : n_ranges(TB, cus_prefill);
  const int64_t R = RA + RB;
  auto bound = [&](int64_t r) -> int64_t {   // first page of range r
    return r <= RA ? r * TA / std::max<int64_t>(RA, 1) : TA + (r - RA) * TB / RB;
  };
  struct Piece { int32_t s, d, k0, k1; };
  std::vector<Piece> pieces;
  std::vector<int32_t> ranges;
  size_t d0 = 0;   // first sequence that can overlap the current range
  for (int64_t r = 0; r < R; ++r) {
    ranges.push_back(int32_t(pieces.size()));
    const int64_t lo_r = bound(r), hi_r = bound(r + 1);
    while (d0 < dec.size() && start[d0 + 1] <= lo_r) ++d0;
    for (size_t d = d0; d < dec.size() && start[d] < hi_r; ++d) {
      const int64_t lo = std::max(lo_r, start[d]), hi = std::min(hi_r, start[d + 1]);
      if (lo >= hi) continue;
      const int32_t s = dec[d];
      pieces.push_back({s, int32_t(d), int32_t((lo - start[d]) * P),
                        int32_t(std::min<int64_t>(seq_lens[s], (hi - start[d]) * P))});
    }
  }
  ranges.push_back(int32_t(pieces.size()));
  const int64_t ppr = std::max(RA ? cdiv(TA, RA) : 0, RB ? cdiv(TB, RB) : 0);   // most pages of a range
  std::vector<int32_t> first_piece(dec.size(), -1), n_pieces(dec.size(), 0);
  for (size_t i = 0; i < pieces.size(); ++i) {
    const int32_t d = pieces[i].d;
    if (first_piece[d] < 0) first_piece[d] = int32_t(i);
    ++n_pieces[d];
  }
  std::vector<int32_t> dec_words;
  int32_t n_split_seqs = 0;
  for (size_t d = 0; d < dec.size(); ++d) n_split_seqs += n_pieces[d] > 1;
  for (size_t i = 0; i < pieces.size(); ++i) {
    const Piece& pc = pieces[i];
    const int32_t item[kItemWords] = {pc.s, int32_t(i) - first_piece[pc.d], n_pieces[pc.d], pc.k0, pc.k1,
                                      first_piece[pc.d], qsl[pc.s], int32_t(i)};
    dec_words.insert(dec_words.end(), item, item + kItemWords);
  }
  const int32_t n_dec_items = int32_t(pieces.size());

  // Prefill tiles of bm rows, the longest causal key range first. A row is
  // a token, or with flat tiles a (token, query head) pair of one KV head,
  // r = token * G + head; a tile's key range ends at the causal limit of its
  // last row's token.
  struct Tile { int32_t s, t, r0, r1, kend; };
  std::vector<Tile> tiles;
  for (int32_t s : pre) {
    const int32_t n = qsl[s + 1] - qsl[s], L = seq_lens[s];
    const int64_t rows = flat ? int64_t(n) * G : n;
    if (rows > INT32_MAX) return set_error(FLEX_ERR_INVALID_ARG, "prefill chunk too long for flat row tiles");
    for (int32_t t = 0; int64_t(t) * bm < rows; ++t) {
      const int32_t r0 = t * bm, r1 = int32_t(std::min<int64_t>(rows, int64_t(t + 1) * bm));
      tiles.push_back({s, t, r0, r1, L - n + (flat ? (r1 - 1) / G + 1 : r1)});
    }
  }
  std::stable_sort(tiles.begin(), tiles.end(), [](const Tile& a, const Tile& b) {
    if (a.kend != b.kend) return a.kend > b.kend;
    if (a.s != b.s) return a.s < b.s;
    return a.t < b.t;
  });

  // Fused order for FLEX_MODE_FUSED (its layout and rule are described with
  // the plan words in host_common.h).
  std::vector<int32_t> fused;
  const bool fusable = !latent && !split && G > 4 && W == 1 && heads_per_wg >= kFusedMinKvHeads && bm == 32;
  if (fusable && (!tiles.empty() || !pieces.empty())) {
    const int64_t rpw = heads_per_wg <= 4 ? 2 : 1;
    const int64_t J = cdiv(R, rpw);
    const int64_t n_pre_wg = int64_t(tiles.size()) * pre_grid_y;
    const double bw_cu = (o.decode_gbps_per_cu != 0.0 ? o.decode_gbps_per_cu : kDefaultDecodeGBpsPerCU) * 1e9;
    const double fl_cu = (o.prefill_tflops_per_cu != 0.0 ? o.prefill_tflops_per_cu : kDefaultPrefillTFlopsPerCU) * 1e12;
    const int64_t chunks = (G + 7) / 8;   // prefill columns per KV head
    // Per XCD: entries and estimated durations (ns) in each phase's order.
    std::vector<int32_t> pe[8], de[8];
    std::vector<int64_t> pd[8], dd[8];
    for (size_t i = 0; i < tiles.size(); ++i) {
      const Tile& t = tiles[i];
      const int64_t rows = t.r1 - t.r0;
      const int64_t pairs = rows * (t.kend - t.r1) + (int64_t(t.r0) + 1 + t.r1) * rows / 2;
      for (int32_t c = 0; c < pre_grid_y; ++c) {
        const int64_t e = int64_t(i) * pre_grid_y + c;
        const int x = 8 % pre_grid_y == 0 ? int(c + pre_grid_y * (int64_t(i) % (8 / pre_grid_y))) : int(e % 8);
        const int64_t heads = std::min<int64_t>(8, G - 8 * (c % chunks));
        const double flops = double(pairs) * double(heads) * double(2 * (sh.head_dim_qk + sh.head_dim_v));
        pe[x].push_back(int32_t(e));
        pd[x].push_back(int64_t(flops / fl_cu * 1e9) + 1);
      }
    }
    const int64_t page_bytes = int64_t(P) * sh.num_kv_heads * (sh.head_dim_qk + sh.head_dim_v) * 2;
    for (int64_t j = 0; j < J; ++j) {
      const int64_t r0 = rpw * j, r1 = std::min(R, rpw * j + rpw);
      const double bytes = double(r1 * T / R - r0 * T / R) * double(page_bytes);
      de[j % 8].push_back(int32_t(n_pre_wg + j));
      dd[j % 8].push_back(int64_t(bytes / bw_cu * 1e9) + 1);
    }
    // Two CU pools per XCD, sized by the plan's CU split (half each when it
    // has none), each handing its phase's work-groups, in order, to its
    // earliest-free CU; entries are listed by simulated start time (prefill
    // first on ties, then phase order).
    const int64_t cap = std::max<int64_t>(2, cus_total / 8);
    int64_t cd = cus_decode < cus_total ? cus_decode * cap / cus_total : cap / 2;
    cd = std::min(cap - 1, std::max<int64_t>(1, cd));
    struct Ev { int64_t start; int kind; size_t k; };
    auto simulate = [](const std::vector<int64_t>& dur, int64_t m, int kind, std::vector<Ev>& out) {
      std::vector<int64_t> free_at(size_t(m), 0);
      for (size_t k = 0; k < dur.size(); ++k) {
        size_t best = 0;
        for (size_t q = 1; q < free_at.size(); ++q)
          if (free_at[q] < free_at[best]) best = q;
        out.push_back({free_at[best], kind, k});
        free_at[best] += dur[k];
      }
    };
    std::vector<int32_t> lists[8];
    size_t longest = 0;
    for (int x = 0; x < 8; ++x) {
      std::vector<Ev> ev;
      simulate(pd[x], de[x].empty() ? cap : cap - cd, 0, ev);
      simulate(dd[x], pe[x].empty() ? cap : cd, 1, ev);
      std::sort(ev.begin(), ev.end(), [](const Ev& a, const Ev& b) {
        if (a.start != b.start) return a.start < b.start;
        if (a.kind != b.kind) return a.kind < b.kind;
        return a.k < b.k;
      });
      for (const Ev& v : ev) lists[x].push_back(v.kind == 0 ? pe[x][v.k] : de[x][v.k]);
      longest = std::max(longest, lists[x].size());
    }
    fused.assign(8 * longest, -1);
    for (int x = 0; x < 8; ++x)
      for (size_t k = 0; k < lists[x].size(); ++k) fused[8 * k + x] = lists[x][k];
  }

  flex_attn_plan_t* plan = new (std::nothrow) flex_attn_plan_t();
  if (!plan) return set_error(FLEX_ERR_INTERNAL, "out of host memory");
  plan->shape = sh;
  plan->rows_per_wg = rows_per_wg;
  plan->cus_total = int32_t(cus_total);
  plan->max_pages_per_seq = max_pages_per_seq;
  const int32_t n_pre_items = int32_t(tiles.size());
  // Launch order for one work-group per piece: longest key range first.
  std::vector<int32_t> order(n_dec_items);
  for (int32_t i = 0; i < n_dec_items; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    return pieces[a].k1 - pieces[a].k0 > pieces[b].k1 - pieces[b].k0;
  });
  std::vector<int32_t> merge_list;   // first piece of every split sequence
  for (size_t d = 0; d < dec.size(); ++d)
    if (n_pieces[d] > 1) merge_list.push_back(first_piece[d]);
  const int32_t off_ranges = kHeaderWords + kItemWords * n_dec_items;
  const int32_t off_order = off_ranges + int32_t(ranges.size());
  const int32_t off_merge = off_order + n_dec_items;
  const int32_t off_pre = off_merge + int32_t(merge_list.size());
  const int32_t off_fused = off_pre + kItemWords * n_pre_items;
  const int32_t off_lens = off_fused + int32_t(fused.size());
  const int32_t total = off_lens + 2 * num_seqs + 1;
  auto& w = plan->words;
  w.assign(kHeaderWords, 0);
  w[H_MAGIC] = kPlanMagic;
  w[H_VERSION] = kPlanVersion;
  w[H_NUM_SEQS] = num_seqs;
  w[H_N_DEC_ITEMS] = n_dec_items;
  w[H_N_PRE_ITEMS] = n_pre_items;
  w[H_N_DEC_SEQS] = int32_t(dec.size());
  w[H_N_PRE_SEQS] = int32_t(pre.size());
  w[H_DEC_WIDTH] = W;
  w[H_PRE_GRID_Y] = pre_grid_y;
  w[H_OFF_DEC] = kHeaderWords;
  w[H_OFF_PRE] = off_pre;
  w[H_PPS] = int32_t(ppr);
  w[H_CUS_DEC] = int32_t(cus_decode);
  w[H_CUS_PRE] = int32_t(cus_prefill);
  w[H_BM] = bm;
  w[H_TOTAL_WORDS] = total;
  w[H_N_RANGES] = int32_t(R);
  w[H_OFF_RANGES] = off_ranges;
  w[H_OFF_ORDER] = off_order;
  w[H_OFF_MERGE] = off_merge;
  w[H_OFF_FUSED] = off_fused;
  w[H_N_FUSED] = int32_t(fused.size());
  w[H_OFF_LENS] = off_lens;
  w[H_N_TAIL_RANGES] = int32_t(RB);
  w.insert(w.end(), dec_words.begin(), dec_words.end());
  w.insert(w.end(), ranges.begin(), ranges.end());
  w.insert(w.end(), order.begin(), order.end());
  w.insert(w.end(), merge_list.begin(), merge_list.end());
  for (const Tile& t : tiles) {
    const int32_t item[kItemWords] = {t.s, t.t, t.r0, t.r1, t.kend, 0, 0, 0};
    w.insert(w.end(), item, item + kItemWords);
  }
  w.insert(w.end(), fused.begin(), fused.end());
  w.insert(w.end(), seq_lens, seq_lens + num_seqs);
  w.insert(w.end(), qsl, qsl + num_seqs + 1);

  // Workspace: per (decode item, column) the rows' (max, sum) pairs, then the
  // unnormalised partial outputs; needed only when some sequence is split.
  size_t ws = 0;
  if (n_split_seqs > 0) {
    const size_t stats = size_t(n_dec_items) * W * rows_per_wg * 2 * 4;
    ws = size_t(cdiv(int64_t(stats), 256) * 256) + size_t(n_dec_items) * W * rows_per_wg * sh.head_dim_v * 4;
  }
  flex_attn_plan_info& info = plan->info;
  std::memset(&info, 0, sizeof(info));
  info.num_seqs = num_seqs;
  info.n_decode_seqs = int32_t(dec.size());
  info.n_prefill_seqs = int32_t(pre.size());
  info.n_decode_items = n_dec_items;
  info.n_prefill_items = n_pre_items;
  info.n_split_seqs = n_split_seqs;
  info.decode_wg_width = W;
  info.prefill_grid_y = pre_grid_y;
  info.pages_per_split = int32_t(ppr);
  info.n_decode_ranges = int32_t(R);
  info.cus_decode = int32_t(cus_decode);
  info.cus_prefill = int32_t(cus_prefill);
  info.bm = bm;
  info.plan_words = total;
  info.device_plan_bytes = size_t(cdiv(int64_t(total) * 4, 256) * 256);
  info.workspace_bytes = ws;
  info.decode_bytes = double(dec_bytes);
  info.prefill_flops = double(pre_flops);
  info.n_fused_wgs = int32_t(fused.size());
  info.n_decode_tail_ranges = int32_t(RB);
  for (size_t i = size_t(ranges[RA]); i < pieces.size(); ++i)
    info.decode_tail_bytes += double(pieces[i].k1 - pieces[i].k0) * double(kv_row);
  if (log_level() > 0) log_plan(*plan);
  *out_plan = plan;
  return FLEX_OK;
}

extern "C" int flex_attn_validate_host(const flex_attn_plan_t* plan, const int32_t* bt, int32_t bt_stride,
                                       int32_t num_pages, const int32_t* h_seq_lens, const int32_t* h_qsl) {
  clear_error();
  if (!plan || !bt || !h_seq_lens || !h_qsl) return set_error(FLEX_ERR_INVALID_ARG, "NULL argument");
  const int32_t B = plan->info.num_seqs;
  const int32_t* lens = plan->words.data() + plan->words[H_OFF_LENS];
  const int32_t* pqsl = lens + B;
  if (bt_stride < plan->max_pages_per_seq)
    return set_error(FLEX_ERR_INVALID_ARG, "block_table_stride " + std::to_string(bt_stride) +
                                               " is below the plan's max_pages_per_seq " +
                                               std::to_string(plan->max_pages_per_seq));
  if (num_pages <= 0) return set_error(FLEX_ERR_INVALID_ARG, "num_pages must be positive");
  const int64_t P = plan->shape.page_size;
  for (int32_t s = 0; s < B; ++s) {
    if (h_seq_lens[s] != lens[s])
      return set_error(FLEX_ERR_INVALID_ARG, "sequence " + std::to_string(s) + ": seq_lens differs from the plan's");
    if (h_qsl[s] != pqsl[s] || (s == B - 1 && h_qsl[B] != pqsl[B]))
      return set_error(FLEX_ERR_INVALID_ARG,
                       "sequence " + std::to_string(s) + ": query_start_loc differs from the plan's");
    for (int64_t t = 0; t < cdiv(lens[s], P); ++t) {
      const int32_t pg = bt[int64_t(s) * bt_stride + t];
      if (pg < 0 || pg >= num_pages)
        return set_error(FLEX_ERR_INVALID_ARG, "sequence " + std::to_string(s) + ", page " + std::to_string(t) +
                                                   ": block-table entry " + std::to_string(pg) +
                                                   " outside [0, num_pages)");
    }
  }
  return FLEX_OK;
}

extern "C" int flex_attn_plan_info_get(const flex_attn_plan_t* plan, flex_attn_plan_info* out) {
  clear_error();
  if (!plan || !out) return set_error(FLEX_ERR_INVALID_ARG, "plan or out is NULL");
  *out = plan->info;
  return FLEX_OK;
}

extern "C" int flex_attn_plan_export(const flex_attn_plan_t* plan, int32_t* h_dst, size_t n_words) {
  clear_error();
  if (!plan || !h_dst) return set_error(FLEX_ERR_INVALID_ARG, "plan or destination is NULL");
  if (n_words < plan->words.size())
    return set_error(FLEX_ERR_WORKSPACE, "destination holds fewer words than the plan");
  std::memcpy(h_dst, plan->words.data(), plan->words.size() * sizeof(int32_t));
  return FLEX_OK;
}

extern "C" void flex_attn_plan_destroy(flex_attn_plan_t* plan) { delete plan; }
