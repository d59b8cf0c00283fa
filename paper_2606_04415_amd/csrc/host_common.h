// Host-side internals shared by the planner and the run calls.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "flexattn.h"

namespace flexattn {

// Plan word layout: a 24-word header, 8 words per decode item, the range
// table (the decode tail's ranges last; H_N_TAIL_RANGES of them), the piece launch order, the merge list, 8 words per prefill item,
// the fused order, then the batch's seq_lens [B] and query_start_loc [B+1]
// as the plan saw them (the debug check compares the device copies with
// them).
constexpr int32_t kPlanMagic = 0x46504C58;
constexpr int32_t kPlanVersion = 7;
constexpr int kHeaderWords = 24;
constexpr int kItemWords = 8;

enum HeaderField {
  H_MAGIC = 0, H_VERSION, H_NUM_SEQS, H_N_DEC_ITEMS, H_N_PRE_ITEMS, H_N_DEC_SEQS,
  H_N_PRE_SEQS, H_DEC_WIDTH, H_PRE_GRID_Y, H_OFF_DEC, H_OFF_PRE, H_PPS, H_CUS_DEC,
  H_CUS_PRE, H_BM, H_TOTAL_WORDS, H_N_RANGES, H_OFF_RANGES, H_OFF_ORDER, H_OFF_MERGE,
  H_OFF_FUSED, H_N_FUSED, H_OFF_LENS, H_N_TAIL_RANGES
};

// Decode item (one piece: the overlap of a balanced page range with one
// sequence) words: seq, rank j of the piece in its sequence, pieces of the
// sequence, key_begin, key_end, workspace slot of the sequence's piece 0,
// the sequence's query token index, this piece's workspace slot (= its list
// index). The range table after the decode items holds the first piece of
// each range, then the piece count; the launch order after it lists the
// pieces by key count descending (ties: slot) for launches of one
// work-group per piece; the merge list after that holds, for each decode
// sequence cut into several pieces (batch order), the index of its first
// piece.
// Prefill item words: seq, tile, row_begin, row_end, key_end, unused x3.
// Fused order (one launch for both phases, FLEX_MODE_FUSED): entry b is the
// work of launch work-group b: e < n_pre_items * prefill_grid_y is prefill
// work-group e (tile e / grid_y, column e % grid_y); e >= that is decode
// work-group j = e - n_pre_items * prefill_grid_y, balanced ranges
// [rpw * j, rpw * j + rpw) (rpw = 2 when a decode work-group covers at most
// 4 KV heads, else 1); -1 is padding. Work-group b runs on XCD b % 8 (the
// dispatcher deals work-groups to XCDs in turn, and within an XCD in id order
// as CUs free up). Prefill column c goes to the XCDs x with x % grid_y == c
// when grid_y divides 8 (as the prefill launch places them), other entries
// to XCD (index % 8). Per XCD the entries are listed by the start time a
// simulation gives them: the XCD's CUs (cus_total / 8) form a prefill pool
// and a decode pool sized by the plan's split (cus_decode / cus_total of
// them decode, half when the plan has no split, at least one each; a phase
// with no work on the XCD leaves the other all of them); each pool hands its
// phase's work-groups, in phase order, to its earliest-free CU (lowest index
// on ties), a work-group lasting its cost-model time in whole ns plus one
// (prefill: 2 (d_qk + d_v) x its query heads x the tile's causal query-key
// pairs / prefill_tflops_per_cu; decode: the ranges' pages x page bytes /
// decode_gbps_per_cu); ties in start time list prefill first, then phase
// order. Empty (0 entries) when the shape has no fused form: grouped-query
// heads, G > 4, 3..8 KV heads, 32-row tiles.
constexpr int kFusedMinKvHeads = 3;

// Most pages one balanced decode range may hold (its block-table entries are
// staged in LDS by the decode kernel).
constexpr int64_t kMaxRangePages = 8192;
// Flat 128-row prefill work-groups resident on one CU (50 KB of LDS each).
constexpr int64_t kFlatResidentPerCu = 3;

// KV heads one grouped-query decode work-group covers (one wave each, or
// several waves per head when fewer heads than 4).
constexpr int32_t kDecodeHeadsPerWG = 8;

// Cost-model rates when the options leave them 0, measured on MI355X with
// the Qwen2.5-7B-shaped mixed step: one CU's decode rate beside a running
// prefill (4.29 TB/s on 96 CUs, 5.21 TB/s on 128), one CU's prefill rate
// (511 TFLOP/s on 128 CUs), and the device's streaming rate (decode alone on
// 160 to 256 CUs: 6.3 to 6.55 TB/s).
constexpr double kDefaultDecodeGBpsPerCU = 43.0;
constexpr double kDefaultPrefillTFlopsPerCU = 4.0;
constexpr double kDefaultHbmGBps = 6500.0;
// Grouped-query prefill time in the cost model: the larger of the work at
// the per-CU rate and the largest work-group's at the rate one work-group
// reaches alone (a 4-wave flat 128-row work-group: about 0.6 of a CU; a
// 32-token work-group of the KV group's query heads: a whole CU), plus a
// launch latency. Fitted to 2048-token chunks on 96 to 160 CUs: prompts of
// 512 to 2048 tokens on prefixes up to 4096 run within 15% of it (the
// work alone missed small chunks by 10 to 60 us).
constexpr double kFlatWgCuShare = 0.6;
constexpr double kPrefillLaunchSec = 10e-6;
// The controller, which sees no tiles, predicts a co-run step with a decode
// tail only when its predicted prefill phase lasts at least this long.
constexpr double kTailMinPrefillUs = 100.0;

// Rows (query heads) one decode work-group owns in the 576/512 layout.
constexpr int kLatentRowsPerWG = 64;       // latent heads must be a multiple of this
constexpr int kLatentRowsPerWGWide = 128;  // heads per latent decode work-group when they divide

int set_error(int status, const std::string& msg);
// Validates an attention shape (sets the error text); FLEX_OK if supported.
int check_shape(const flex_attn_shape& sh);
void clear_error();
int log_level();

}  // namespace flexattn

struct flex_attn_plan {
  flex_attn_shape shape;
  flex_attn_plan_info info;
  int32_t cus_total;        // the CU count the plan was partitioned against
  int32_t rows_per_wg;      // query rows of one decode work-group
  int32_t max_pages_per_seq;  // block-table entries a row must hold
  std::vector<int32_t> words;
};

namespace flexattn {
void log_plan(const ::flex_attn_plan_t& p);
}  // namespace flexattn
