// Host-side internals shared by the planner and the run calls.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "flexattn.h"

namespace flexattn {

// Plan word layout: a 16-word header, then 8 words per decode item, then 8
// words per prefill item.
constexpr int32_t kPlanMagic = 0x46504C58;
constexpr int32_t kPlanVersion = 4;
constexpr int kHeaderWords = 20;
constexpr int kItemWords = 8;

enum HeaderField {
  H_MAGIC = 0, H_VERSION, H_NUM_SEQS, H_N_DEC_ITEMS, H_N_PRE_ITEMS, H_N_DEC_SEQS,
  H_N_PRE_SEQS, H_DEC_WIDTH, H_PRE_GRID_Y, H_OFF_DEC, H_OFF_PRE, H_PPS, H_CUS_DEC,
  H_CUS_PRE, H_BM, H_TOTAL_WORDS, H_N_RANGES, H_OFF_RANGES, H_OFF_ORDER, H_OFF_MERGE
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

// Most pages one balanced decode range may hold (its block-table entries are
// staged in LDS by the decode kernel).
constexpr int64_t kMaxRangePages = 8192;

// KV heads one grouped-query decode work-group covers (one wave each, or
// several waves per head when fewer heads than 4).
constexpr int32_t kDecodeHeadsPerWG = 8;

// Rows (query heads) one decode work-group owns in the 576/512 layout.
constexpr int kLatentRowsPerWG = 64;       // latent heads must be a multiple of this
constexpr int kLatentRowsPerWGWide = 128;  // heads per latent decode work-group when they divide

int set_error(int status, const std::string& msg);
// Validates an attention shape (sets the error text); FLEX_OK if supported.
int check_shape(const flex_attn_shape& sh);
void clear_error();

}  // namespace flexattn

struct flex_attn_plan {
  flex_attn_shape shape;
  flex_attn_plan_info info;
  int32_t cus_total;        // the CU count the plan was partitioned against
  int32_t rows_per_wg;      // query rows of one decode work-group
  std::vector<int32_t> words;
};
