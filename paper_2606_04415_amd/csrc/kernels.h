// Kernel parameter blocks and launchers (host-callable, defined in attention.hip
// and kv_append.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace flexattn {

struct CacheRef {
  const uint16_t* base;
  int64_t sp, ss, sh;  // element strides: page, slot, kv head
};

struct AttnParams {
  const uint16_t* q;
  CacheRef kc, vc;
  const int32_t* bt;
  int32_t bt_stride;
  const int32_t* seq_lens;
  const int32_t* qsl;
  uint16_t* out;
  float* lse;
  const int32_t* items;   // device pointer to the first item of this phase
  int32_t n_items;
  const int32_t* ranges;  // decode: first piece of each balanced range (+ the piece count)
  const int32_t* order;   // decode: pieces longest first, for one work-group per piece
  const int32_t* merge;   // decode: first piece of every split sequence
  int32_t n_merge;
  int32_t n_ranges;
  int32_t range_pages;    // decode: most pages a range holds
  float* ws_stats;        // decode: [item][W][rows][2] (max in log2 units, sum)
  float* ws_o;            // decode: [item][W][rows][d_v] unnormalised partial outputs
  int32_t Hq, Hkv, G;     // G = query heads per KV head
  int32_t P;
  int32_t rows_per_wg;    // decode rows owned by one work-group
  int32_t grid_y;
  int32_t xcd_remap;      // prefill: 1-D grid mapped so each XCD serves one column
  float scale_log2;       // sm_scale * log2(e)
};

hipError_t launch_decode(const AttnParams& p, int head_dim_qk, bool has_splits, hipStream_t stream);
// The split-K merge alone (after decode launches that skipped it).
hipError_t launch_decode_merge(const AttnParams& p, int head_dim_qk, hipStream_t stream);
hipError_t launch_prefill(const AttnParams& p, int head_dim_qk, int bm, hipStream_t stream);
// One launch for both phases (grouped-query heads, 32-row prefill tiles):
// pp / pd are the prefill and decode parameter blocks, order the plan's fused
// order (n_order entries), then the split-K merge when has_splits.
hipError_t launch_fused(const AttnParams& pp, const AttnParams& pd, const int32_t* order, int n_order,
                        int head_dim_qk, int ranges_per_wg, bool has_splits, hipStream_t stream);
hipError_t launch_gather(const CacheRef& kc, const CacheRef& vc, bool has_v, const int32_t* bt_row,
                         int32_t L, int32_t P, int32_t Hkv, int32_t dqk, int32_t dv,
                         uint16_t* k_out, uint16_t* v_out, hipStream_t stream);
hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream);

// Debug check of one run's device metadata against the plan's own copy of
// the lengths (plan_lens: seq_lens [B] then query_start_loc [B+1], on the
// device): every sequence's seq_lens and query_start_loc entry equal to the
// plan's, and block-table entries 0 .. ceil(L_s / P) - 1 of every row in
// [0, num_pages). Enqueues the check on stream, waits for it, and returns in
// *kind 0 (all good) or the first violation found (1: seq_lens, 2:
// query_start_loc, 3: block-table entry) and in *seq its sequence.
hipError_t debug_check(const int32_t* seq_lens, const int32_t* qsl, const int32_t* bt, int32_t bt_stride,
                       const int32_t* plan_lens, int32_t num_seqs, int32_t P, int32_t num_pages, int32_t* kind,
                       int32_t* seq, hipStream_t stream);

struct AppendParams {
  const uint16_t* k_new;
  const uint16_t* v_new;
  int64_t k_new_stride, v_new_stride;   // elements per token row
  const int32_t* slot_mapping;
  int64_t n_tokens;
  CacheRef kc, vc;                      // destinations (base cast back to writable)
  int64_t num_slots;                    // num_pages * P
  int32_t P;
  int32_t dk, dv;                       // head dimensions of the copied rows (dv unused when ck only)
  int64_t ck, cv;                       // 16-byte chunks per token: Hkv*dk/8 and Hkv*dv/8 (0 if aliased)
  int32_t* bad_count;                   // optional: tokens whose slot lies outside the pool
};

hipError_t launch_kv_append(const AppendParams& a, hipStream_t stream);

}  // namespace flexattn
