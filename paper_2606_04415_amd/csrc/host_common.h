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
constexpr int32_t kPlanVersion = 2;
constexpr int kHeaderWords = 16;
constexpr int kItemWords = 8;

enum HeaderField {
  H_MAGIC = 0, H_VERSION, H_NUM_SEQS, H_N_DEC_ITEMS, H_N_PRE_ITEMS, H_N_DEC_SEQS,
  H_N_PRE_SEQS, H_DEC_WIDTH, H_PRE_GRID_Y, H_OFF_DEC, H_OFF_PRE, H_PPS, H_CUS_DEC,
  H_CUS_PRE, H_BM, H_TOTAL_WORDS
};

// Decode item words: seq, split, n_splits, key_begin, key_end, workspace slot
// of the sequence's split 0, decode-sequence ordinal, this item's workspace
// slot. Items are in launch order (longest key range first); slots are in
// batch order, so split j of a sequence sits at slot 0 + j.
// Prefill item words: seq, tile, row_begin, row_end, key_end, unused x3.

// Rows (query heads) one decode work-group owns in the 576/512 layout.
constexpr int kLatentRowsPerWG = 64;

int set_error(int status, const std::string& msg);
void clear_error();

}  // namespace flexattn

struct flex_attn_plan {
  flex_attn_shape shape;
  flex_attn_plan_info info;
  int32_t rows_per_wg;      // query rows of one decode work-group
  std::vector<int32_t> words;
};
