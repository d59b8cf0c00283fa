/*
 * flexattn: mixed prefill/decode paged attention on one MI355X (gfx950).
 *
 * What the library computes. FlexNPU co-locates the prefill and decode phases
 * of LLM serving on one device and schedules them by phase: prefill is
 * compute-intensive, decode is bound by memory bandwidth and KV-cache reads,
 * and both read one shared KV pool (Abstract; Sec. 1; Sec. 3; Sec. 3.3;
 * Sec. 3.4 "Phase-Aware Dispatch", "Memory Locality"). The data-parallel work
 * inside such a co-located step is attention over one mixed batch:
 *
 *   for sequence s with n_s new query tokens and L_s keys (0 <= n_s <= L_s),
 *   query i sits at absolute position L_s - n_s + i and attends keys
 *   0 .. L_s - n_s + i (bottom-right causal alignment; decode is n_s = 1);
 *   key t of s is row (block_table[s][t / P], t % P) of the paged caches;
 *   query head h reads KV head h / (Hq / Hkv);
 *   out = softmax(sm_scale * q K^T) V,  lse = log-sum-exp of the scaled scores
 *   (natural log).
 *
 * The paper writes none of this down (it defines no kernel); the definition
 * is textbook scaled dot-product attention. Where the paper leaves a detail
 * open, this library reads it as: pages laid out [page][slot][kv_head][dim];
 * bottom-right causal alignment; consecutive query heads share a KV head;
 * bf16 inputs, fp32 accumulation and softmax, bf16 output rounded to nearest
 * even.
 *
 * Conventions for every call:
 *  - Every call returns an int status (FLEX_OK or a negative FLEX_ERR_*);
 *    nothing throws across this boundary. flex_attn_last_error() returns a
 *    thread-local text describing the last failure on the calling thread.
 *  - Device memory is owned by the caller; the library never allocates
 *    device memory (its only device state is fixed module memory: the step
 *    counters of co-run pairs, the scratch of flex_attn_mixed_static and the
 *    debug check's status word). Host plan objects and co-run pairs are
 *    owned by the library until their destroy call.
 *  - Run calls (decode, prefill, mixed, debug gather, workspace init) only
 *    enqueue work on the given HIP stream (a hipStream_t passed as void*;
 *    NULL is the null stream) and return; they never synchronise.
 *  - Tensors are bf16 with the innermost dimension contiguous; every base
 *    pointer and every row stride must be a multiple of 16 bytes.
 */
#ifndef FLEXATTN_H
#define FLEXATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define FLEX_OK 0
#define FLEX_ERR_INVALID_ARG (-1)  /* malformed metadata, null/misaligned pointer, inconsistent args */
#define FLEX_ERR_UNSUPPORTED (-2)  /* well-formed but outside the supported shapes */
#define FLEX_ERR_WORKSPACE (-3)    /* device plan or workspace buffer too small */
#define FLEX_ERR_HIP (-4)          /* a HIP runtime call failed; text in flex_attn_last_error() */
#define FLEX_ERR_INTERNAL (-5)

/* Modes of flex_attn_mixed. */
#define FLEX_MODE_SERIAL 0  /* prefill then decode on the caller stream, all CUs */
#define FLEX_MODE_CORUN 1   /* prefill and decode on two CU-masked streams, joined */
#define FLEX_MODE_FUSED 2   /* one launch holding both phases' work-groups, interleaved */

/* Attention geometry of one layer.
 * Supported:
 *  - (head_dim_qk, head_dim_v) in {(64,64), (128,128)} with
 *    num_q_heads / num_kv_heads <= 16, page_size 16 or 64 (grouped-query);
 *  - (576, 512) with v_aliases_k = 1, num_kv_heads = 1 and num_q_heads a
 *    multiple of 64, page_size 16 or 64 (absorbed latent attention: the
 *    value row of a key is the first 512 columns of its 576-wide key row);
 *  - (192, 128) with v_aliases_k = 0, num_q_heads / num_kv_heads <= 16 and
 *    page_size 64 (latent attention with its heads split out: keys 128 + 64
 *    rope, values 128 per head). This layout is prefill only: every sequence
 *    with one or more new tokens is a prefill sequence.
 * sm_scale must be finite and > 0. */
typedef struct flex_attn_shape {
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim_qk;
  int32_t head_dim_v;
  int32_t page_size;
  float sm_scale;
  int32_t v_aliases_k;
} flex_attn_shape;

/* Planner tunables; a zero field takes the default in brackets.
 * cus_decode: CUs the decode phase is partitioned for and, in co-run mode,
 * runs on [0 = all]; -1 asks the cost model to choose the split among
 * multiples of split_granule from the rates below. */
typedef struct flex_attn_plan_opts {
  int32_t cus_total;          /* [256] */
  int32_t cus_decode;         /* CUs of the co-run decode share [0 = all CUs: no share];
                                 -1: the cost model's best multiple of split_granule */
  int32_t bm;                 /* prefill rows per tile. Grouped-query: 16 or 32 tokens, or 128
                                 flattened rows, each a (token, query head) pair of one KV head
                                 [128 when the batch gives every prefill CU at least four
                                 such 128-row work-groups, or, on a co-run share, when all of
                                 them fit in one round (three per CU); else 32]; 576/512: 64
                                 or 128 tokens [128]; 192/128: 128 [128] */
  int32_t min_split_tokens;   /* shortest balanced decode range, in keys [256] */
  int32_t wg_per_cu;          /* decode work-groups aimed at per CU
                                 [1 grouped-query, 2 for 576/512] */
  int32_t split_granule;      /* co-run split granularity in CUs [32] */
  double hbm_gbps;            /* cost model: device streaming rate [6500, what decode
                                 reaches on 160 to 256 CUs] */
  double decode_gbps_per_cu;  /* cost model: decode bandwidth one CU draws beside a running
                                 prefill [43] */
  double prefill_tflops_per_cu; /* cost model: prefill rate of one CU [4] (defaults measured
                                   on MI355X, the Qwen2.5-7B-shaped mixed step). Grouped-query
                                   prefill time: the larger of the work at this rate and the
                                   largest work-group's (its rows x every key of its sequence)
                                   at 0.6 of it (flat 128-row tiles) or all of it (32-token
                                   tiles), plus 10 us */
  int32_t decode_tail;        /* 0: a grouped-query co-run plan whose decode share would
                                 outlast the prefill (cost model) splits its decode pages in
                                 two groups of ranges, the second (the tail) run on the
                                 prefill stream after the prefill (see flex_attn_mixed);
                                 -1: no tail [0] */
} flex_attn_plan_opts;

/* Summary of a plan. */
typedef struct flex_attn_plan_info {
  int32_t num_seqs;
  int32_t n_decode_seqs;     /* sequences with one new token (none in the 192/128 layout) */
  int32_t n_prefill_seqs;    /* sequences with two or more new tokens (one or more: 192/128) */
  int32_t n_decode_items;    /* decode pieces: (sequence, key range) work items */
  int32_t n_prefill_items;   /* (sequence, row tile) work items */
  int32_t n_split_seqs;      /* decode sequences cut into more than one piece */
  int32_t decode_wg_width;   /* work-groups per decode range or piece (grid y) */
  int32_t n_decode_ranges;   /* balanced page ranges the decode pieces form */
  int32_t prefill_grid_y;    /* work-groups per prefill tile (grid y) */
  int32_t pages_per_split;   /* pages per decode range (rounded up) */
  int32_t cus_decode;
  int32_t cus_prefill;
  int32_t bm;
  int32_t plan_words;        /* int32 words in the exported / uploaded plan */
  size_t device_plan_bytes;  /* bytes the device copy of the plan needs */
  size_t workspace_bytes;    /* bytes of workspace decode needs (0 if none) */
  double decode_bytes;       /* algorithmic KV bytes of the decode phase */
  double prefill_flops;      /* algorithmic flops of the prefill phase */
  int32_t n_fused_wgs;       /* work-groups of the one-launch (FUSED) form; 0 when the
                                shape has none (see flex_attn_mixed) */
  int32_t n_decode_tail_ranges; /* the last ranges of the n_decode_ranges, which CORUN runs
                                   on the prefill stream after the prefill; 0: no tail */
  double decode_tail_bytes;  /* algorithmic KV bytes of those ranges (the CORUN decode
                                phase streams decode_bytes - decode_tail_bytes) */
} flex_attn_plan_info;

/* Device tensors of one run. Strides are in elements.
 *  (A run call checks pointers, alignment, strides, block_table_stride >=
 *  the plan's max_pages_per_seq and buffer sizes; the contents of
 *  block_table, seq_lens and query_start_loc are checked only in debug mode,
 *  see flex_attn_set_debug, or on the host by flex_attn_validate_host.)
 *  q        bf16 [T, Hq, d_qk], contiguous (T = query_start_loc[B]).
 *  k_cache  bf16 pages: element (page, slot, kv_head, d) at
 *           page*k_stride[0] + slot*k_stride[1] + kv_head*k_stride[2] + d.
 *  v_cache  same with v_stride and d < d_v; ignored (may be NULL) when the
 *           shape has v_aliases_k.
 *           For both caches the page stride and page_size * slot stride must
 *           each stay below 2^31 bytes (kernels address within a page with
 *           32-bit offsets); larger strides are FLEX_ERR_INVALID_ARG.
 *  block_table int32 [B, >= max_pages_per_seq], row stride block_table_stride;
 *           entries 0 .. ceil(L_s / P) - 1 of row s must lie in [0, num_pages).
 *  seq_lens int32 [B], query_start_loc int32 [B+1]: the same values the plan
 *           was built from (a mismatch is undefined behaviour).
 *  out      bf16 [T, Hq, d_v], contiguous; rows of sequences with n_s = 0 are
 *           untouched.
 *  lse      fp32 [T, Hq] or NULL.
 *  d_plan   the plan uploaded with flex_attn_plan_upload.
 *  workspace  device scratch of >= flex_attn_plan_info.workspace_bytes (may
 *           be NULL when that is 0): the split decode items' partial results,
 *           written by the decode kernel and read by the merge kernel that
 *           follows it on the same stream. Its contents need no
 *           initialisation. Two runs in flight at once must not share a
 *           workspace. */
typedef struct flex_attn_args {
  const void* q;
  const void* k_cache;
  const void* v_cache;
  int64_t k_stride[3];
  int64_t v_stride[3];
  int32_t num_pages;
  const int32_t* block_table;
  int32_t block_table_stride;
  const int32_t* seq_lens;
  const int32_t* query_start_loc;
  void* out;
  float* lse;
  const void* d_plan;
  size_t d_plan_bytes;
  void* workspace;
  size_t workspace_bytes;
} flex_attn_args;

typedef struct flex_attn_plan flex_attn_plan_t;
typedef struct flex_attn_corun flex_attn_corun_t;

/* Text of a status code (static storage). */
const char* flex_attn_status_string(int status);
/* Detail of the last failure on this thread (thread-local, valid until the next call). */
const char* flex_attn_last_error(void);

/* Build a host plan: validate the integer metadata, classify each sequence by
 * its new-token count (1 -> decode, >= 2 -> prefill, 0 -> nothing; in the
 * (192, 128) layout every count >= 1 is prefill), split each
 * decode sequence's keys into page-aligned ranges, tile each prefill chunk into
 * rows, longest key range first, and fix the co-run CU split. This mirrors the
 * daemon's validate-then-enqueue step and its per-phase queues (Sec. 3.2;
 * Sec. 3.4 "Phase-Aware Dispatch"). Host only: makes no HIP call.
 * h_query_start_loc [num_seqs+1] and h_seq_lens [num_seqs] are host arrays.
 * opts may be NULL (defaults). On success *out_plan owns a new plan.
 * Errors: FLEX_ERR_INVALID_ARG (query_start_loc[0] != 0 or decreasing, n_s > L_s,
 * L_s > max_pages_per_seq * page_size, Hq % Hkv != 0, bad scale, bad opts,
 * null pointers), FLEX_ERR_UNSUPPORTED (shape outside the supported set). */
int flex_attn_plan(const flex_attn_shape* shape, const flex_attn_plan_opts* opts,
                   int32_t num_seqs, const int32_t* h_query_start_loc,
                   const int32_t* h_seq_lens, int32_t max_pages_per_seq,
                   flex_attn_plan_t** out_plan);

/* Check one run's metadata on the host against the plan, before copying it
 * to the device: block_table_stride >= the plan's max_pages_per_seq, entries
 * 0 .. ceil(L_s / P) - 1 of every block-table row in [0, num_pages), and
 * h_seq_lens [B] / h_query_start_loc [B+1] equal to the values the plan was
 * built from. FLEX_OK, or FLEX_ERR_INVALID_ARG naming the first violation.
 * Host arrays only; no HIP call. */
int flex_attn_validate_host(const flex_attn_plan_t* plan, const int32_t* h_block_table,
                            int32_t block_table_stride, int32_t num_pages, const int32_t* h_seq_lens,
                            const int32_t* h_query_start_loc);

/* Debug mode of the run calls, the device-side counterpart of
 * flex_attn_validate_host (the paper's daemon validates each request before
 * dispatch, Sec. 3.2). With level 1, flex_attn_decode, _prefill, _mixed and
 * _mixed_static first run a check kernel on the stream that compares the
 * device seq_lens and query_start_loc with the plan's copy (uploaded with
 * the plan) and every block-table entry a sequence uses with
 * [0, num_pages); they wait for it (the call then synchronises the stream,
 * so debug mode does not suit graph capture) and return
 * FLEX_ERR_INVALID_ARG naming the sequence without launching attention
 * when a check fails. Level 0 turns it off. The initial level is 1 when the
 * environment variable FLEX_ATTN_DEBUG is set to anything but 0 when the
 * library loads, else 0. Returns the previous level, or FLEX_ERR_INVALID_ARG
 * for a negative level. FLEX_ATTN_LOG=1 in the environment prints one line
 * per plan on stderr (2: also every work item). */
int flex_attn_set_debug(int level);

/* Copy the plan summary into *out. */
int flex_attn_plan_info_get(const flex_attn_plan_t* plan, flex_attn_plan_info* out);

/* Copy the plan's int32 words (header, decode items, prefill items) to host
 * memory h_dst of n_words >= plan_words; FLEX_ERR_WORKSPACE if too small. */
int flex_attn_plan_export(const flex_attn_plan_t* plan, int32_t* h_dst, size_t n_words);

/* Enqueue an H2D copy of the plan words into device buffer d_dst of
 * dst_bytes >= device_plan_bytes on stream. The plan must outlive the copy. */
int flex_attn_plan_upload(const flex_attn_plan_t* plan, void* d_dst, size_t dst_bytes, void* stream);

void flex_attn_plan_destroy(flex_attn_plan_t* plan);

/* Decode phase (sequences with one new token; the 192/128 layout has none):
 * split-K attention over each
 * sequence's pages, streamed from HBM, then (when some sequence is split) a
 * second launch that merges the splits in split order:
 * out = sum_j e^{m_j - M} O_j / sum_j e^{m_j - M} l_j, M = max_j m_j. */
int flex_attn_decode(const flex_attn_plan_t* plan, const flex_attn_args* args, void* stream);

/* Prefill phase (sequences with two or more new tokens, or one or more in the
 * 192/128 layout): causal flash
 * attention over key tiles gathered through block_table into LDS, with QK^T
 * and PV on bf16 matrix cores and fp32 accumulation. */
int flex_attn_prefill(const flex_attn_plan_t* plan, const flex_attn_args* args, void* stream);

/* One mixed step: both phases of the plan. FLEX_MODE_SERIAL runs prefill then
 * decode on stream; FLEX_MODE_CORUN forks stream into the two CU-masked
 * streams of corun (prefill on its prefill stream, decode on its decode
 * stream) and joins them back into stream, the one-device analog of the
 * paper's dynamic co-location (Sec. 3.4). When the plan has a decode tail
 * (info n_decode_tail_ranges > 0), the decode stream runs the other ranges
 * and the prefill stream runs the tail's ranges right after the prefill, so
 * the prefill share streams decode pages once its own phase is done; the
 * split-K merge then runs on stream after the join. The fork and, for steps expected
 * to run under a millisecond (plan info work on the pair's CU shares), the
 * join are stream memory operations on the pair's step counters; longer
 * steps join through events, which hold no CU while they wait (a memory-value
 * wait on stream polls from a kernel). FLEX_MODE_FUSED runs both phases
 * in one launch on stream (then the split-K merge): each work-group of the
 * launch serves one prefill work-group's tile and column or one or two
 * decode ranges, in the plan's fused order (the phases interleaved by a
 * simulated dispatch onto a prefill and a decode share of each XCD); the
 * device's dispatcher hands work-groups to compute units as they free up, so
 * the phases share the device without CU masks (the alternative to two
 * streams; an analog of the dispatch-controlled sharing the paper relies on
 * where the device offers no spatial partitioning, Sec. 3 and Sec. 3.4).
 * FUSED needs a plan with n_fused_wgs > 0: grouped-query
 * heads with G = Hq / Hkv > 4, 3 <= Hkv <= 8 and 32-row tiles; otherwise it
 * returns FLEX_ERR_UNSUPPORTED. Outputs are bit-identical between the three
 * modes for the same plan. corun is ignored by FUSED. For SERIAL, corun may
 * be NULL; if given, it is used only for phase timing
 * (flex_attn_corun_set_timing). For CORUN, pass a
 * stream of your own, not HIP's legacy default (NULL) stream: that stream
 * synchronizes implicitly with the pair's streams, which stalls the host at
 * every step (measured: 230 us of host time per step instead of 24). */
int flex_attn_mixed(const flex_attn_plan_t* plan, const flex_attn_args* args, int mode,
                    void* stream, flex_attn_corun_t* corun);

/* Allocation-free form of flex_attn_mixed, for callers that cannot allocate
 * device memory or let a library call do so: code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation. Same arguments,
 * modes, kernels and results (bit-identical to flex_attn_mixed for the same
 * plan and inputs), except that the decode phase's split-K partials go to a
 * fixed scratch array the library holds in device memory (one per device it
 * runs on, kept until the process ends) instead of args->workspace, whose two
 * fields are ignored. The call itself allocates nothing.
 * Limit: the plan's workspace_bytes must not exceed
 * flex_attn_static_scratch_bytes() (32 MiB), else FLEX_ERR_WORKSPACE with the
 * sizes in flex_attn_last_error(). The scratch needs no initialisation and
 * keeps the last call's contents. Every call on one device shares that
 * device's scratch: two calls whose work can overlap on one GPU (different
 * streams, or a co-run step still running) race; issue them in order on one
 * stream. The first call on a device resolves the scratch address
 * (hipGetSymbolAddress); a failure there is FLEX_ERR_HIP. */
int flex_attn_mixed_static(const flex_attn_plan_t* plan, const flex_attn_args* args, int mode,
                           void* stream, flex_attn_corun_t* corun);
/* Bytes of the allocation-free call's scratch array. */
size_t flex_attn_static_scratch_bytes(void);

/* Create two streams on the current device, restricted by CU masks to
 * cus_prefill and cus_decode compute units (disjoint; each eighth of the
 * device holds one CU of every shader engine of every XCD, so any split keeps
 * the engines evenly equipped), and a 24-byte device buffer of step counters through which
 * flex_attn_mixed forks and joins them (stream memory writes and waits). Each
 * count must be a positive multiple of an eighth of the device's CUs (32 on
 * a 256-CU MI355X) and their sum at most the device's CU count. One pair
 * serves one host thread at a time. Keep few pairs open per process: HIP
 * serves a process's streams from a small pool of hardware queues
 * (GPU_MAX_HW_QUEUES, 4 by default), so with several pairs open the two
 * streams of one pair can share a queue and its phases then run one after
 * the other (measured: co-run steps 1.6 times longer with seven pairs open
 * than with one); to change the split, destroy the pair and create another. */
int flex_attn_corun_create(int32_t cus_prefill, int32_t cus_decode, flex_attn_corun_t** out);
/* Synchronizes the device (no stream may still wait on the counters), then
 * frees the pair. */
void flex_attn_corun_destroy(flex_attn_corun_t* corun);
/* The two streams (hipStream_t) of a co-run pair. */
int flex_attn_corun_streams(const flex_attn_corun_t* corun, void** prefill_stream, void** decode_stream);

/* Per-phase timing, the runtime profile the paper's scheduler consumes
 * (operator execution time per phase, Sec. 3.3). With timing enabled, every
 * flex_attn_mixed call given this corun object (in either mode) records HIP
 * events around each phase's kernel on the stream that kernel runs on, into
 * a ring of FLEX_TIMING_RING steps. Enabling clears the ring. */
#define FLEX_TIMING_RING 1024
int flex_attn_corun_set_timing(flex_attn_corun_t* corun, int enable);
/* Wait for the recorded steps and copy their phase durations in milliseconds
 * (oldest first; a phase with no work reads 0) into prefill_ms / decode_ms of
 * capacity max_steps each; *n_steps receives the count copied. */
int flex_attn_corun_timing_read(flex_attn_corun_t* corun, float* prefill_ms, float* decode_ms,
                                int32_t max_steps, int32_t* n_steps);

/* Test aid: copy the L_s key rows (and value rows unless v_aliases_k) of
 * sequence seq, gathered through block_table with a plain per-element page
 * lookup (row t from page block_table[seq][t / P], slot t % P, the paging
 * contract above), into contiguous k_out [L_s, Hkv, d_qk] and
 * v_out [L_s, Hkv, d_v] (bf16). It checks the caller's block table and
 * strides against the contract; it does not run the attention kernels' own
 * address paths (those load through page windows staged in LDS and buffer
 * resources per page). seq_len is L_s on the host. */
int flex_attn_debug_gather(const flex_attn_plan_t* plan, const flex_attn_args* args, int32_t seq,
                           int32_t seq_len, void* k_out, void* v_out, void* stream);

/* Zero a buffer (e.g. a workspace) on stream with a fill kernel; bytes must
 * be a multiple of 4. No run call requires it. */
int flex_attn_workspace_init(void* workspace, size_t bytes, void* stream);

/* KV append: the write side of the KV pool both phases share (Sec. 3.4,
 * "Memory Locality": co-located prefill and decode extend and read one pool
 * in place instead of moving KV caches between workers). Token t's key row
 * (and value row unless the shape has v_aliases_k) is copied into slot
 * slot_mapping[t] of the paged caches: page slot / page_size, row
 * slot % page_size, the same addressing the attention calls read through
 * block_table. Typically called for a step's new tokens before the step's
 * attention, on the same stream.
 *  k_new        bf16 [n_tokens][Hkv][d_qk]: token t's row starts at element
 *               t * k_new_stride; the Hkv*d_qk values of a row are contiguous.
 *  v_new        bf16 [n_tokens][Hkv][d_v] with v_new_stride; ignored (may be
 *               NULL) when the shape has v_aliases_k.
 *  slot_mapping int32 [n_tokens], device: a negative entry skips its token
 *               (padding); an entry >= num_pages * page_size also skips it and
 *               adds 1 to *bad_count when bad_count is not NULL (device int32,
 *               not reset by the call). Two tokens given one slot leave one of
 *               the two rows there (unspecified which).
 *  k_cache, k_stride, v_cache, v_stride, num_pages: as in flex_attn_args; the
 *               caches are written.
 * Pointers and row strides must be 16-byte multiples; n_tokens >= 0 (0 launches
 * nothing). Enqueues one kernel on stream and returns. */
typedef struct flex_attn_append_args {
  const void* k_new;
  const void* v_new;
  int64_t k_new_stride;
  int64_t v_new_stride;
  const int32_t* slot_mapping;
  int64_t n_tokens;
  void* k_cache;
  int64_t k_stride[3];
  void* v_cache;
  int64_t v_stride[3];
  int64_t num_pages;
  int32_t* bad_count;
} flex_attn_append_args;

int flex_attn_kv_append(const flex_attn_shape* shape, const flex_attn_append_args* args, void* stream);

/* ------------------------------------------------------------------------
 * Online co-location controller (host only, no HIP call).
 *
 * Sec. 3.4 "Phase-Aware Dispatch": the runtime watches (1) pending prefill and
 * decode work, (2) recent per-phase execution times, (3) memory-bandwidth
 * pressure, (4) decode progress and the active sequence count and (5)
 * device utilisation, and moves the prefill/decode balance step by step:
 * when decode is close to saturating bandwidth, more compute units would not
 * speed it up, so prefill gets them; when decode work backs up, decode's
 * share grows. Sec. 3.3: the per-phase profile it uses is coarse and updated
 * continuously during execution.
 *
 * Here the balance is the CU split of the next co-run step (or serial
 * execution). The controller keeps, per candidate split, a running estimate
 * of each phase's rate in that split (decode GB/s, prefill TFLOP/s), seeded
 * by a prior (flex_ctl_set_profile, else the cost model of the options) and
 * updated from every observed step (exponentially weighted). For the next
 * step it predicts each split's time, max(B / decode rate, F / prefill rate)
 * + a co-run overhead, and serial time B / rate + F / rate, then applies the
 * rule above among the co-run splits within `tolerance` of the best
 * prediction: decode backlog (pending_decode_seqs >= backlog_seqs) takes the
 * largest decode share; otherwise decode bandwidth pressure (the last
 * observed decode rate reached sat_frac of hbm_gbps) or a prefill backlog
 * (pending_prefill_tokens >= backlog_prefill_tokens) takes the smallest;
 * otherwise the best prediction. Serial runs when it is predicted fastest or
 * one phase has no work. When the step has a one-launch form (FLEX_MODE_FUSED)
 * its prediction is the serial prediction times a running ratio of observed
 * fused to observed serial step times (prior fused_prior; see
 * flex_ctl_observation); it is chosen
 * when strictly below both the serial and the best co-run prediction. Every
 * explore_every-th decision tries a neighbouring split instead of a co-run
 * choice, and every fourth such turn tries the one-launch form instead of
 * the choice when it has one and was not chosen, so stale estimates are
 * refreshed. Signal (5), utilisation, enters through the observations: a
 * split whose phases finish unevenly leaves CUs idle and shows up as a
 * slower observed rate.
 * ---------------------------------------------------------------------- */
typedef struct flex_ctl flex_ctl_t;

/* A zero field takes the default in brackets (use a tiny positive value for
 * a tolerance or overhead of zero). */
typedef struct flex_ctl_opts {
  int32_t cus_total;            /* [256] */
  int32_t granule;              /* candidate splits are multiples [64]; must divide cus_total */
  int32_t explore_every;        /* [16]; a negative value disables exploration */
  int32_t backlog_seqs;         /* decode backlog that raises decode's share [256] */
  int32_t backlog_prefill_tokens; /* prefill backlog that lowers it [8192] */
  double alpha;                 /* weight of a new observation (0, 1] [0.25] */
  double tolerance;             /* relative band around the best prediction [0.03] */
  double sat_frac;              /* bandwidth-pressure threshold, fraction of hbm_gbps [0.6] */
  double hbm_gbps;              /* [8000] */
  double corun_overhead_us;     /* fork/join cost added to co-run predictions [10] */
  double decode_gbps_per_cu;    /* prior when no profile is set [60] */
  double prefill_tflops_per_cu; /* prior when no profile is set [5] */
  double fused_prior;           /* prior of (one-launch step time) / (serial step time) [0.9] */
} flex_ctl_opts;

/* Signals describing the step about to run and the queues behind it. */
typedef struct flex_ctl_signals {
  double decode_bytes;          /* algorithmic KV bytes of the step's decode phase (plan info) */
  double prefill_flops;         /* algorithmic flops of its prefill phase (plan info) */
  int32_t pending_prefill_tokens; /* (1) prompt tokens still waiting for prefill */
  int32_t pending_decode_seqs;  /* (1)/(4) sequences waiting to decode beyond this step */
  int32_t active_decode_seqs;   /* (4) sequences decoding in this step */
  int32_t fused_available;      /* the step's plan has a one-launch form (n_fused_wgs > 0) */
  int32_t decode_tail;          /* co-run plans of this step form a decode tail (grouped-query
                                   heads, plan option decode_tail 0): a co-run split whose
                                   predicted prefill lasts 100 us or more is then predicted as
                                   the prefill plus decode's rest at the rate decode reaches on
                                   all CUs, not as the slower phase */
} flex_ctl_signals;

/* What the last step measured (e.g. flex_attn_corun_timing_read). A
 * one-launch (FUSED) step has no separate phase times: set fused = 1 and
 * step_ms to its duration (cus_decode, decode_ms and prefill_ms are then
 * ignored). The controller keeps the ratio of such steps' durations to its
 * serial prediction for the same work, and the same ratio for serial steps
 * that report step_ms (0: not reported), and predicts a fused step as the
 * serial prediction times the first ratio over the second, so that launch
 * and gap costs outside the phase times weigh on both alike. */
typedef struct flex_ctl_observation {
  int32_t cus_decode;           /* split it ran with; 0 or cus_total = serial */
  double decode_bytes, prefill_flops;
  double decode_ms, prefill_ms; /* phase durations (0 for a phase with no work) */
  int32_t fused;                /* 1: the step ran as one launch */
  double step_ms;               /* the step's duration: required for fused steps, optional
                                   for serial ones (0 = not reported) */
} flex_ctl_observation;

#define FLEX_CTL_ONE_PHASE 0      /* one phase has no work: serial */
#define FLEX_CTL_BEST 1           /* best predicted split */
#define FLEX_CTL_SERIAL_FASTER 2  /* serial predicted fastest */
#define FLEX_CTL_BACKLOG 3        /* decode backlog: largest decode share in the band */
#define FLEX_CTL_BW_SATURATED 4   /* bandwidth pressure: smallest decode share in the band */
#define FLEX_CTL_EXPLORE 5        /* neighbour of the choice, to refresh its estimate */
#define FLEX_CTL_PREFILL_BACKLOG 6 /* prefill backlog: smallest decode share in the band */
#define FLEX_CTL_FUSED_FASTER 7   /* the one-launch form predicted fastest */

typedef struct flex_ctl_decision {
  int32_t mode;                 /* FLEX_MODE_SERIAL, FLEX_MODE_CORUN or FLEX_MODE_FUSED */
  int32_t cus_decode;           /* co-run: decode CUs (plan opts cus_decode); serial: cus_total */
  int32_t cus_prefill;
  int32_t reason;               /* FLEX_CTL_* */
  double predicted_us;          /* predicted step time of the returned choice */
} flex_ctl_decision;

int flex_ctl_create(const flex_ctl_opts* opts, flex_ctl_t** out);
void flex_ctl_destroy(flex_ctl_t* ctl);
/* Seed the estimates from a measured profile (Sec. 3.3), e.g. the CU sweep:
 * n points of (cus, decode GB/s alone on cus CUs, prefill TFLOP/s alone on cus
 * CUs), cus ascending multiples of the granule; rates between points are
 * interpolated linearly, and a split's co-run estimate starts at the alone
 * rates of its two shares. Resets every estimate. */
int flex_ctl_set_profile(flex_ctl_t* ctl, int32_t n, const int32_t* cus, const double* decode_gbps,
                         const double* prefill_tflops);
int flex_ctl_observe(flex_ctl_t* ctl, const flex_ctl_observation* obs);
int flex_ctl_decide(flex_ctl_t* ctl, const flex_ctl_signals* sig, flex_ctl_decision* out);
/* Current estimates: for each decode share k * granule (k = 1 .. K - 1,
 * K = cus_total / granule) the co-run decode GB/s and prefill TFLOP/s of that
 * split, then the serial pair; K entries each, capacity >= K. */
int flex_ctl_estimates(const flex_ctl_t* ctl, double* decode_gbps, double* prefill_tflops, int32_t capacity);

/* ------------------------------------------------------------------------
 * Time-slice scheduler: temporal multiplexing of the phases instead of CU
 * partitioning (Sec. 3 and Sec. 3.4: when the device offers no spatial
 * partitioning, each phase's execution share is enforced by dispatch control
 * and phase-aware temporal multiplexing; Sec. 4: the prefill/decode
 * time-slice ratio is the knob of the serving experiments).
 *
 * Each step runs one phase alone on the whole device (flex_attn_decode or
 * flex_attn_prefill on a batch holding only that phase). The scheduler keeps
 * the device time spent in each phase, both totals multiplied by `decay`
 * before every new observation is added (a window of about 1 / (1 - decay)
 * steps; decay 1 keeps the whole history), and picks the next step's phase:
 * the only ready phase if one is ready; with both ready, decode when
 * decode_ms * (1 - decode_share) <= prefill_ms * decode_share (decode's
 * share of the windowed time is at or below its target, ties to decode),
 * else prefill. Over a run with both phases always ready and decay 1, decode's
 * time stays within one longest step of decode_share times the total time
 * (so its share is within that step's duration over the total of the
 * target). Host-only; no HIP call.
 * ---------------------------------------------------------------------- */
typedef struct flex_ts flex_ts_t;

/* A zero field takes the default in brackets. */
typedef struct flex_ts_opts {
  double decode_share;          /* target fraction of device time for decode, in (0, 1) [0.5] */
  double decay;                 /* weight kept by past time at each observation, in (0, 1] [1] */
} flex_ts_opts;

#define FLEX_TS_DECODE 0
#define FLEX_TS_PREFILL 1

int flex_ts_create(const flex_ts_opts* opts, flex_ts_t** out);
void flex_ts_destroy(flex_ts_t* ts);
/* Next step's phase (FLEX_TS_DECODE or FLEX_TS_PREFILL) into *phase.
 * FLEX_ERR_INVALID_ARG when neither phase is ready. */
int flex_ts_next(const flex_ts_t* ts, int32_t decode_ready, int32_t prefill_ready, int32_t* phase);
/* A finished step: its phase and duration (ms, >= 0). */
int flex_ts_observe(flex_ts_t* ts, int32_t phase, double ms);
/* The windowed device time of each phase (ms). */
int flex_ts_totals(const flex_ts_t* ts, double* decode_ms, double* prefill_ms);

#ifdef __cplusplus
}
#endif
#endif /* FLEXATTN_H */
