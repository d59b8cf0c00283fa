// Run calls of the C ABI: argument checks, kernel parameter blocks, serial and
// co-run launch, plan upload, debug gather, workspace fill and KV append.
//
// Co-run is the one-device analog of the paper's dynamic prefill/decode
// co-location (Sec. 3.4): the two phases of one step share the device and its
// KV pool, each restricted to its own set of compute units through a CU-masked
// stream, instead of running back to back on all units.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "host_common.h"
#include "kernels.h"

using namespace flexattn;

struct flex_attn_corun {
  hipStream_t prefill = nullptr;
  hipStream_t decode = nullptr;
  // Fork/join through stream memory operations on three 64-bit step counters
  // (caller, prefill, decode): far cheaper, on the host and on the device,
  // than event records and event waits across queues, for sub-millisecond
  // steps; longer steps join through events (see run_mixed). The counters
  // only ever compare greater-or-equal, so steps of either kind mix.
  uint64_t* flags = nullptr;   // a slot of the device's counter pool, zeroed at creation
  int slot = -1;
  uint64_t step = 0;           // last step number issued
  int device = 0;
  int cus_prefill = 0;
  int cus_decode = 0;
  // phase timing ring: events around each phase's kernel, per recorded step
  bool timing = false;
  int64_t t_count = 0;
  std::vector<hipEvent_t> ev;        // 4 per slot: prefill start/end, decode start/end
  std::vector<unsigned char> has;    // 2 per slot: prefill ran, decode ran
  hipEvent_t join_ev[2] = {nullptr, nullptr};   // prefill done, decode done (long steps)
};

namespace {

int hip_fail(hipError_t e, const char* what) {
  return set_error(FLEX_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Checks shared by every run call; fills the kernel parameter block. A
// non-NULL ws_override (of at least the plan's workspace_bytes) replaces the
// caller's workspace, whose fields are then ignored.
int prepare(const flex_attn_plan_t* plan, const flex_attn_args* a, AttnParams* p, void* ws_override = nullptr) {
  if (!plan || !a) return set_error(FLEX_ERR_INVALID_ARG, "plan or args is NULL");
  const flex_attn_shape& sh = plan->shape;
  const flex_attn_plan_info& info = plan->info;
  const bool has_work = info.n_decode_items + info.n_prefill_items > 0;
  std::memset(p, 0, sizeof(*p));
  if (!has_work) return FLEX_OK;
  if (!a->q || !a->k_cache || !a->block_table || !a->seq_lens || !a->query_start_loc || !a->out || !a->d_plan)
    return set_error(FLEX_ERR_INVALID_ARG, "a required device pointer is NULL");
  const void* v = sh.v_aliases_k ? a->k_cache : a->v_cache;
  if (!v) return set_error(FLEX_ERR_INVALID_ARG, "v_cache is NULL");
  if (!aligned16(a->q) || !aligned16(a->k_cache) || !aligned16(v) || !aligned16(a->out) || !aligned16(a->d_plan))
    return set_error(FLEX_ERR_INVALID_ARG, "q, caches, out and d_plan must be 16-byte aligned");
  const int64_t* vs = sh.v_aliases_k ? a->k_stride : a->v_stride;
  for (int i = 0; i < 3; ++i) {
    if (a->k_stride[i] <= 0 || vs[i] <= 0 || (a->k_stride[i] * 2) % 16 || (vs[i] * 2) % 16)
      return set_error(FLEX_ERR_INVALID_ARG, "cache strides must be positive multiples of 16 bytes");
  }
  // Within a page the kernels use 32-bit byte offsets.
  const int64_t lim = int64_t(1) << 31;
  if (a->k_stride[0] * 2 >= lim || vs[0] * 2 >= lim || a->k_stride[1] * 2 * sh.page_size >= lim ||
      vs[1] * 2 * sh.page_size >= lim)
    return set_error(FLEX_ERR_INVALID_ARG, "cache page stride or page_size * slot stride reaches 2^31 bytes");
  if (a->k_stride[2] < sh.head_dim_qk || vs[2] < (sh.v_aliases_k ? sh.head_dim_qk : sh.head_dim_v))
    return set_error(FLEX_ERR_INVALID_ARG, "cache head stride smaller than the head dimension");
  if (a->num_pages <= 0) return set_error(FLEX_ERR_INVALID_ARG, "num_pages must be positive");
  if (a->block_table_stride < 1 || a->block_table_stride < plan->max_pages_per_seq)
    return set_error(FLEX_ERR_INVALID_ARG, "block_table_stride " + std::to_string(a->block_table_stride) +
                                               " is below the plan's max_pages_per_seq " +
                                               std::to_string(plan->max_pages_per_seq));
  if (a->d_plan_bytes < info.device_plan_bytes)
    return set_error(FLEX_ERR_WORKSPACE, "d_plan_bytes smaller than the plan's device_plan_bytes");
  if (info.workspace_bytes > 0 && !ws_override) {
    if (!a->workspace) return set_error(FLEX_ERR_INVALID_ARG, "workspace is NULL");
    if (!aligned16(a->workspace)) return set_error(FLEX_ERR_INVALID_ARG, "workspace must be 16-byte aligned");
    if (a->workspace_bytes < info.workspace_bytes)
      return set_error(FLEX_ERR_WORKSPACE, "workspace_bytes smaller than the plan's workspace_bytes");
  }
  p->q = static_cast<const uint16_t*>(a->q);
  p->kc = CacheRef{static_cast<const uint16_t*>(a->k_cache), a->k_stride[0], a->k_stride[1], a->k_stride[2]};
  p->vc = CacheRef{static_cast<const uint16_t*>(v), vs[0], vs[1], vs[2]};
  p->bt = a->block_table;
  p->bt_stride = a->block_table_stride;
  p->seq_lens = a->seq_lens;
  p->qsl = a->query_start_loc;
  p->out = static_cast<uint16_t*>(a->out);
  p->lse = a->lse;
  p->Hq = sh.num_q_heads;
  p->Hkv = sh.num_kv_heads;
  p->G = sh.num_q_heads / sh.num_kv_heads;
  p->P = sh.page_size;
  p->rows_per_wg = plan->rows_per_wg;
  p->scale_log2 = sh.sm_scale * 1.4426950408889634f;
  if (info.workspace_bytes > 0) {
    const int32_t W = info.decode_wg_width;
    const size_t stats = size_t(info.n_decode_items) * W * plan->rows_per_wg * 2 * 4;
    char* ws = static_cast<char*>(ws_override ? ws_override : a->workspace);
    p->ws_stats = reinterpret_cast<float*>(ws);
    p->ws_o = reinterpret_cast<float*>(ws + ((stats + 255) / 256) * 256);
  }
  return FLEX_OK;
}

// Debug mode (flex_attn_set_debug, or FLEX_ATTN_DEBUG=1 in the environment
// when the library loads): before any attention launch, a check kernel
// compares the device seq_lens / query_start_loc with the plan's copy and
// every used block-table entry with [0, num_pages); a violation is
// FLEX_ERR_INVALID_ARG and nothing is launched.
std::atomic<int> g_debug{[] {
  const char* v = std::getenv("FLEX_ATTN_DEBUG");
  return v && *v && std::strcmp(v, "0") != 0 ? 1 : 0;
}()};

int debug_validate(const flex_attn_plan_t* plan, const flex_attn_args* a, hipStream_t s) {
  if (g_debug.load(std::memory_order_relaxed) == 0) return FLEX_OK;
  const flex_attn_plan_info& info = plan->info;
  if (info.n_decode_items + info.n_prefill_items == 0) return FLEX_OK;
  int32_t kind = 0, seq = -1;
  const hipError_t e =
      debug_check(a->seq_lens, a->query_start_loc, a->block_table, a->block_table_stride,
                  static_cast<const int32_t*>(a->d_plan) + plan->words[H_OFF_LENS], info.num_seqs,
                  plan->shape.page_size, a->num_pages, &kind, &seq, s);
  if (e != hipSuccess) return hip_fail(e, "debug check");
  static const char* what[] = {"", "device seq_lens differs from the plan's", "device query_start_loc differs "
                               "from the plan's", "a block-table entry lies outside [0, num_pages)"};
  if (kind != 0)
    return set_error(FLEX_ERR_INVALID_ARG, "debug check, sequence " + std::to_string(seq) + ": " +
                                               what[kind >= 1 && kind <= 3 ? kind : 0]);
  return FLEX_OK;
}

// Which decode ranges a launch covers: all of them (then the merge), or the
// co-run decode share's part / the tail (no merge; it follows the join).
enum class DecodePart { all, head, tail };

int run_decode(const flex_attn_plan_t* plan, AttnParams p, const flex_attn_args* a, hipStream_t s,
               DecodePart part = DecodePart::all) {
  const flex_attn_plan_info& info = plan->info;
  if (info.n_decode_items == 0) return FLEX_OK;
  const int32_t R = plan->words[H_N_RANGES], RB = plan->words[H_N_TAIL_RANGES];
  p.items = static_cast<const int32_t*>(a->d_plan) + plan->words[H_OFF_DEC];
  p.n_items = info.n_decode_items;
  p.ranges = static_cast<const int32_t*>(a->d_plan) + plan->words[H_OFF_RANGES];
  p.n_ranges = part == DecodePart::all ? R : part == DecodePart::head ? R - RB : RB;
  if (part == DecodePart::tail) p.ranges += R - RB;   // (a range reads entries r and r + 1)
  p.order = static_cast<const int32_t*>(a->d_plan) + plan->words[H_OFF_ORDER];
  p.merge = static_cast<const int32_t*>(a->d_plan) + plan->words[H_OFF_MERGE];
  p.n_merge = info.n_split_seqs;
  p.range_pages = info.pages_per_split;
  p.grid_y = info.decode_wg_width;
  if (p.n_ranges == 0) return FLEX_OK;
  const hipError_t e =
      launch_decode(p, plan->shape.head_dim_qk, part == DecodePart::all && info.n_split_seqs > 0, s);
  return e == hipSuccess ? FLEX_OK : hip_fail(e, "decode launch");
}

int run_decode_merge(const flex_attn_plan_t* plan, AttnParams p, const flex_attn_args* a, hipStream_t s) {
  const flex_attn_plan_info& info = plan->info;
  if (info.n_decode_items == 0 || info.n_split_seqs == 0) return FLEX_OK;
  p.items = static_cast<const int32_t*>(a->d_plan) + plan->words[H_OFF_DEC];
  p.n_items = info.n_decode_items;
  p.merge = static_cast<const int32_t*>(a->d_plan) + plan->words[H_OFF_MERGE];
  p.n_merge = info.n_split_seqs;
  p.grid_y = info.decode_wg_width;
  const hipError_t e = launch_decode_merge(p, plan->shape.head_dim_qk, s);
  return e == hipSuccess ? FLEX_OK : hip_fail(e, "merge launch");
}

int run_prefill(const flex_attn_plan_t* plan, AttnParams p, const flex_attn_args* a, hipStream_t s) {
  const flex_attn_plan_info& info = plan->info;
  if (info.n_prefill_items == 0) return FLEX_OK;
  p.items = static_cast<const int32_t*>(a->d_plan) + plan->words[H_OFF_PRE];
  p.n_items = info.n_prefill_items;
  p.grid_y = info.prefill_grid_y;
  const hipError_t e = launch_prefill(p, plan->shape.head_dim_qk, info.bm, s);
  return e == hipSuccess ? FLEX_OK : hip_fail(e, "prefill launch");
}

// Both phases in one launch through the plan's fused order.
int run_fused(const flex_attn_plan_t* plan, const AttnParams& p, const flex_attn_args* a, hipStream_t s) {
  const flex_attn_plan_info& info = plan->info;
  if (info.n_prefill_items + info.n_decode_items == 0) return FLEX_OK;
  const int32_t n = plan->words[H_N_FUSED];
  if (n == 0)
    return set_error(FLEX_ERR_UNSUPPORTED,
                     "no one-launch form for this plan (needs grouped-query heads, G > 4, 3..8 KV heads, bm 32)");
  const int32_t* d = static_cast<const int32_t*>(a->d_plan);
  AttnParams pp = p, pd = p;
  pp.items = d + plan->words[H_OFF_PRE];
  pp.n_items = info.n_prefill_items;
  pp.grid_y = info.prefill_grid_y;
  pd.items = d + plan->words[H_OFF_DEC];
  pd.n_items = info.n_decode_items;
  pd.ranges = d + plan->words[H_OFF_RANGES];
  pd.n_ranges = plan->words[H_N_RANGES];
  pd.order = d + plan->words[H_OFF_ORDER];
  pd.merge = d + plan->words[H_OFF_MERGE];
  pd.n_merge = info.n_split_seqs;
  pd.range_pages = info.pages_per_split;
  pd.grid_y = info.decode_wg_width;
  const int heads_per_wg = plan->rows_per_wg / p.G;
  const hipError_t e = launch_fused(pp, pd, d + plan->words[H_OFF_FUSED], n, plan->shape.head_dim_qk,
                                    heads_per_wg <= 4 ? 2 : 1, info.n_split_seqs > 0, s);
  return e == hipSuccess ? FLEX_OK : hip_fail(e, "fused launch");
}

// Step counters of the co-run pairs: a fixed pool of slots (3 counters
// each, padded to 4) per device in module memory, so creating a pair
// allocates no device memory. Host code uses the address resolved per device
// with hipGetSymbolAddress, never the array's name.
constexpr int kCorunSlots = 64;
static __device__ __align__(256) uint64_t corun_counters[kCorunSlots * 4];
std::mutex g_corun_mu;
uint64_t* g_corun_base[64] = {};
bool g_corun_used[64][kCorunSlots] = {};

int corun_slot_acquire(int dev, int* slot, uint64_t** flags) {
  if (dev < 0 || dev >= 64) return set_error(FLEX_ERR_UNSUPPORTED, "device index beyond the counter table");
  std::lock_guard<std::mutex> lock(g_corun_mu);
  if (!g_corun_base[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(corun_counters));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(corun_counters)");
    g_corun_base[dev] = static_cast<uint64_t*>(ptr);
  }
  for (int i = 0; i < kCorunSlots; ++i) {
    if (!g_corun_used[dev][i]) {
      g_corun_used[dev][i] = true;
      *slot = i;
      *flags = g_corun_base[dev] + 4 * i;
      return FLEX_OK;
    }
  }
  return set_error(FLEX_ERR_UNSUPPORTED, "more than " + std::to_string(kCorunSlots) + " co-run pairs on one device");
}

void corun_slot_release(int dev, int slot) {
  if (dev < 0 || dev >= 64 || slot < 0) return;
  std::lock_guard<std::mutex> lock(g_corun_mu);
  g_corun_used[dev][slot] = false;
}

// CU masks in eighths of the device. On MI355X (8 XCDs x 4 shader engines x 8
// CUs) mask bit i selects a CU of XCD i % 8, shader engine (i >> 3) & 3,
// position i >> 5 within the engine (measured by recording the hardware ids
// of the work-groups each mask admits). Eighth k is the 32-bit word k: one CU
// of every shader engine of every XCD. Work-groups are handed to XCDs and to
// engines in turn, so a phase runs as fast as its least-equipped engine: any
// set of eighths keeps the engines equal (a mask that fills some engines and
// half-fills others ran no faster than the half-filled engines allow).
int eighth_of(int i) { return i >> 5; }

void build_mask(int lo_eighth, int eighths, int total, uint32_t* mask, int words) {
  for (int i = 0; i < words; ++i) mask[i] = 0;
  for (int i = 0; i < total; ++i) {
    const int e = eighth_of(i % 256);
    if (e >= lo_eighth && e < lo_eighth + eighths) mask[i >> 5] |= 1u << (i & 31);
  }
}

// Launch one phase, bracketed by timing events when the co-run object asks for them.
template <typename Fn>
int timed_phase(flex_attn_corun* c, int phase, bool has_work, hipStream_t s, Fn&& launch) {
  if (!c || !c->timing || !has_work) return launch(s);
  const int64_t slot = c->t_count % FLEX_TIMING_RING;
  hipError_t e = hipEventRecord(c->ev[slot * 4 + 2 * phase], s);
  if (e != hipSuccess) return hip_fail(e, "timing record");
  const int st = launch(s);
  if (st != FLEX_OK) return st;
  if ((e = hipEventRecord(c->ev[slot * 4 + 2 * phase + 1], s)) != hipSuccess) return hip_fail(e, "timing record");
  c->has[slot * 2 + phase] = 1;
  return FLEX_OK;
}

void timing_begin_step(flex_attn_corun* c) {
  if (!c || !c->timing) return;
  const int64_t slot = c->t_count % FLEX_TIMING_RING;
  c->has[slot * 2] = c->has[slot * 2 + 1] = 0;
}

void timing_end_step(flex_attn_corun* c) {
  if (c && c->timing) ++c->t_count;
}

}  // namespace

extern "C" int flex_attn_plan_upload(const flex_attn_plan_t* plan, void* d_dst, size_t dst_bytes, void* stream) {
  clear_error();
  if (!plan || !d_dst) return set_error(FLEX_ERR_INVALID_ARG, "plan or destination is NULL");
  const size_t bytes = plan->words.size() * sizeof(int32_t);
  if (dst_bytes < bytes) return set_error(FLEX_ERR_WORKSPACE, "destination smaller than the plan");
  const hipError_t e = hipMemcpyAsync(d_dst, plan->words.data(), bytes, hipMemcpyHostToDevice,
                                      static_cast<hipStream_t>(stream));
  return e == hipSuccess ? FLEX_OK : hip_fail(e, "plan upload");
}

extern "C" int flex_attn_decode(const flex_attn_plan_t* plan, const flex_attn_args* args, void* stream) {
  clear_error();
  AttnParams p;
  int st = prepare(plan, args, &p);
  if (st != FLEX_OK) return st;
  if ((st = debug_validate(plan, args, static_cast<hipStream_t>(stream))) != FLEX_OK) return st;
  return run_decode(plan, p, args, static_cast<hipStream_t>(stream));
}

extern "C" int flex_attn_prefill(const flex_attn_plan_t* plan, const flex_attn_args* args, void* stream) {
  clear_error();
  AttnParams p;
  int st = prepare(plan, args, &p);
  if (st != FLEX_OK) return st;
  if ((st = debug_validate(plan, args, static_cast<hipStream_t>(stream))) != FLEX_OK) return st;
  return run_prefill(plan, p, args, static_cast<hipStream_t>(stream));
}

namespace {

// Whether a co-run step of this plan is expected to run for a millisecond or
// more (longer phase on its CU share, at about 1 PFLOP/s of prefill and
// 6 TB/s of decode per 256 CUs). Such steps join through events.
constexpr double kEventJoinUs = 1000.0;
bool long_step(const flex_attn_plan_t* plan, const flex_attn_corun* c) {
  const double pre_us = plan->info.prefill_flops / (1.0e15 / 256.0 * c->cus_prefill) * 1e6;
  const double dec_us = plan->info.decode_bytes / (6.0e12 / 256.0 * c->cus_decode) * 1e6;
  return std::max(pre_us, dec_us) >= kEventJoinUs;
}

int run_mixed(const flex_attn_plan_t* plan, const flex_attn_args* args, int mode, void* stream,
              flex_attn_corun_t* corun, void* ws_override) {
  if (mode != FLEX_MODE_SERIAL && mode != FLEX_MODE_CORUN && mode != FLEX_MODE_FUSED)
    return set_error(FLEX_ERR_INVALID_ARG, "unknown mode");
  AttnParams p;
  int st = prepare(plan, args, &p, ws_override);
  if (st != FLEX_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = debug_validate(plan, args, s)) != FLEX_OK) return st;
  if (mode == FLEX_MODE_FUSED) return run_fused(plan, p, args, s);
  const bool has_pre = plan->info.n_prefill_items > 0, has_dec = plan->info.n_decode_items > 0;
  auto pre = [&](hipStream_t ps) { return run_prefill(plan, p, args, ps); };
  auto dec = [&](hipStream_t ds) { return run_decode(plan, p, args, ds); };
  if (mode == FLEX_MODE_SERIAL) {
    timing_begin_step(corun);
    st = timed_phase(corun, 0, has_pre, s, pre);
    if (st != FLEX_OK) return st;
    st = timed_phase(corun, 1, has_dec, s, dec);
    if (st != FLEX_OK) return st;
    timing_end_step(corun);
    return FLEX_OK;
  }
  if (!corun) return set_error(FLEX_ERR_INVALID_ARG, "co-run mode needs a co-run stream pair");
  if (has_pre && has_dec && plan->info.cus_decode != corun->cus_decode)
    return set_error(FLEX_ERR_INVALID_ARG, "the plan's decode phase is partitioned for " +
                                               std::to_string(plan->info.cus_decode) + " CUs, the co-run pair gives it " +
                                               std::to_string(corun->cus_decode));
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != corun->device) return set_error(FLEX_ERR_INVALID_ARG, "co-run pair belongs to another device");
  // Fork: the caller stream publishes the step number once its earlier work
  // is done; both phase streams wait for it. Join: each phase stream
  // publishes the step number after its kernels; the caller stream waits for
  // both.
  const uint64_t step = ++corun->step;
  uint64_t* f = corun->flags;
  if ((e = hipStreamWriteValue64(s, f, step, 0)) != hipSuccess) return hip_fail(e, "fork write");
  if ((e = hipStreamWaitValue64(corun->prefill, f, step, hipStreamWaitValueGte, ~0ull)) != hipSuccess)
    return hip_fail(e, "fork wait");
  if ((e = hipStreamWaitValue64(corun->decode, f, step, hipStreamWaitValueGte, ~0ull)) != hipSuccess)
    return hip_fail(e, "fork wait");
  // With a decode tail, the decode stream takes the other ranges and the
  // prefill stream the tail's, behind the prefill (outside its timed phase);
  // the merge follows the join.
  const bool tail = has_dec && plan->words[H_N_TAIL_RANGES] > 0;
  auto dec_head = [&](hipStream_t ds) { return run_decode(plan, p, args, ds, DecodePart::head); };
  timing_begin_step(corun);
  st = timed_phase(corun, 0, has_pre, corun->prefill, pre);
  if (st != FLEX_OK) return st;
  if (tail && (st = run_decode(plan, p, args, corun->prefill, DecodePart::tail)) != FLEX_OK) return st;
  st = tail ? timed_phase(corun, 1, has_dec, corun->decode, dec_head) : timed_phase(corun, 1, has_dec, corun->decode, dec);
  if (st != FLEX_OK) return st;
  timing_end_step(corun);
  auto merge_after_join = [&]() { return tail ? run_decode_merge(plan, p, args, s) : FLEX_OK; };
  if (long_step(plan, corun)) {
    // The runtime serves a memory-value wait on the caller stream with a
    // polling kernel that may run on any CU for the whole step: over
    // millisecond phases it measured to slow a latent prefill phase by 7%
    // (128 of 256 CUs) to 40% (64 CUs) and to end up to 6 ms after it.
    // Event waits hold no CU; they cost about 12 us more per step.
    if ((e = hipEventRecord(corun->join_ev[0], corun->prefill)) != hipSuccess) return hip_fail(e, "join record");
    if ((e = hipEventRecord(corun->join_ev[1], corun->decode)) != hipSuccess) return hip_fail(e, "join record");
    if ((e = hipStreamWaitEvent(s, corun->join_ev[0], 0)) != hipSuccess) return hip_fail(e, "join wait");
    if ((e = hipStreamWaitEvent(s, corun->join_ev[1], 0)) != hipSuccess) return hip_fail(e, "join wait");
    return merge_after_join();
  }
  if ((e = hipStreamWriteValue64(corun->prefill, f + 1, step, 0)) != hipSuccess) return hip_fail(e, "join write");
  if ((e = hipStreamWriteValue64(corun->decode, f + 2, step, 0)) != hipSuccess) return hip_fail(e, "join write");
  if ((e = hipStreamWaitValue64(s, f + 1, step, hipStreamWaitValueGte, ~0ull)) != hipSuccess)
    return hip_fail(e, "join wait");
  if ((e = hipStreamWaitValue64(s, f + 2, step, hipStreamWaitValueGte, ~0ull)) != hipSuccess)
    return hip_fail(e, "join wait");
  return merge_after_join();
}

// Scratch of the allocation-free entry point: split-K partials of the
// decode phase, one array per device the library runs on (each device holds
// its own copy at its own address), resolved once per device with
// hipGetSymbolAddress. Host code uses only the resolved address: the array's
// name is a host-side stand-in, not a device address.
constexpr size_t kStaticScratchBytes = size_t(32) << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return set_error(FLEX_ERR_UNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if ((e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch))) != hipSuccess)
      return hip_fail(e, "hipGetSymbolAddress(scratch)");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return FLEX_OK;
}

}  // namespace

extern "C" int flex_attn_mixed(const flex_attn_plan_t* plan, const flex_attn_args* args, int mode, void* stream,
                               flex_attn_corun_t* corun) {
  clear_error();
  return run_mixed(plan, args, mode, stream, corun, nullptr);
}

extern "C" int flex_attn_mixed_static(const flex_attn_plan_t* plan, const flex_attn_args* args, int mode,
                                      void* stream, flex_attn_corun_t* corun) {
  clear_error();
  if (!plan || !args) return set_error(FLEX_ERR_INVALID_ARG, "plan or args is NULL");
  if (plan->info.workspace_bytes > kStaticScratchBytes)
    return set_error(FLEX_ERR_WORKSPACE, "the plan needs " + std::to_string(plan->info.workspace_bytes) +
                                             " bytes of split-K scratch; the allocation-free call holds " +
                                             std::to_string(kStaticScratchBytes));
  void* ws = nullptr;
  if (plan->info.workspace_bytes > 0) {
    const int st = static_scratch(&ws);
    if (st != FLEX_OK) return st;
  }
  return run_mixed(plan, args, mode, stream, corun, ws);
}

extern "C" size_t flex_attn_static_scratch_bytes(void) { return kStaticScratchBytes; }

extern "C" int flex_attn_set_debug(int level) {
  clear_error();
  if (level < 0) return set_error(FLEX_ERR_INVALID_ARG, "debug level < 0");
  const int prev = g_debug.exchange(level > 0 ? 1 : 0);
  return prev;
}

extern "C" int flex_attn_corun_create(int32_t cus_prefill, int32_t cus_decode, flex_attn_corun_t** out) {
  clear_error();
  if (!out) return set_error(FLEX_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  hipDeviceProp_t prop;
  if ((e = hipGetDeviceProperties(&prop, dev)) != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
  const int total = prop.multiProcessorCount;
  if (total % 256)
    return set_error(FLEX_ERR_UNSUPPORTED, "co-run needs a device whose CU count is a multiple of 256");
  const int per_eighth = total / 8;
  if (cus_prefill <= 0 || cus_decode <= 0 || cus_prefill % per_eighth || cus_decode % per_eighth ||
      cus_prefill + cus_decode > total)
    return set_error(FLEX_ERR_UNSUPPORTED, "co-run CU counts must be positive multiples of " +
                                               std::to_string(per_eighth) + " summing to at most " +
                                               std::to_string(total));
  const int words = (total + 31) / 32;
  uint32_t mask_p[64], mask_d[64];
  if (words > 64) return set_error(FLEX_ERR_UNSUPPORTED, "too many CUs");
  // Decode takes the low eighths, prefill the next ones.
  build_mask(0, cus_decode / per_eighth, total, mask_d, words);
  build_mask(cus_decode / per_eighth, cus_prefill / per_eighth, total, mask_p, words);
  flex_attn_corun* c = new (std::nothrow) flex_attn_corun();
  if (!c) return set_error(FLEX_ERR_INTERNAL, "out of host memory");
  c->device = dev;
  c->cus_prefill = cus_prefill;
  c->cus_decode = cus_decode;
  if (const int st = corun_slot_acquire(dev, &c->slot, &c->flags); st != FLEX_OK) {
    delete c;
    return st;
  }
  if ((e = hipExtStreamCreateWithCUMask(&c->prefill, words, mask_p)) != hipSuccess ||
      (e = hipExtStreamCreateWithCUMask(&c->decode, words, mask_d)) != hipSuccess ||
      (e = hipMemset(c->flags, 0, 3 * sizeof(uint64_t))) != hipSuccess ||
      (e = hipEventCreateWithFlags(&c->join_ev[0], hipEventDisableTiming)) != hipSuccess ||
      (e = hipEventCreateWithFlags(&c->join_ev[1], hipEventDisableTiming)) != hipSuccess) {
    const int st = hip_fail(e, "co-run stream creation");
    flex_attn_corun_destroy(c);
    return st;
  }
  *out = c;
  return FLEX_OK;
}

extern "C" void flex_attn_corun_destroy(flex_attn_corun_t* c) {
  if (!c) return;
  for (hipEvent_t e : c->ev) (void)hipEventDestroy(e);
  for (hipEvent_t e : c->join_ev)
    if (e) (void)hipEventDestroy(e);
  if (c->prefill) (void)hipStreamDestroy(c->prefill);
  if (c->decode) (void)hipStreamDestroy(c->decode);
  if (c->slot >= 0) {
    (void)hipDeviceSynchronize();   // no stream may still wait on the counters
    corun_slot_release(c->device, c->slot);
  }
  delete c;
}

extern "C" int flex_attn_corun_streams(const flex_attn_corun_t* c, void** p, void** d) {
  clear_error();
  if (!c || !p || !d) return set_error(FLEX_ERR_INVALID_ARG, "NULL argument");
  *p = c->prefill;
  *d = c->decode;
  return FLEX_OK;
}

extern "C" int flex_attn_corun_set_timing(flex_attn_corun_t* c, int enable) {
  clear_error();
  if (!c) return set_error(FLEX_ERR_INVALID_ARG, "corun is NULL");
  if (enable && c->ev.empty()) {
    c->ev.assign(size_t(FLEX_TIMING_RING) * 4, nullptr);
    for (auto& e : c->ev) {
      const hipError_t r = hipEventCreate(&e);
      if (r != hipSuccess) return hip_fail(r, "timing event creation");
    }
    c->has.assign(size_t(FLEX_TIMING_RING) * 2, 0);
  }
  c->timing = enable != 0;
  c->t_count = 0;
  return FLEX_OK;
}

extern "C" int flex_attn_corun_timing_read(flex_attn_corun_t* c, float* prefill_ms, float* decode_ms,
                                           int32_t max_steps, int32_t* n_steps) {
  clear_error();
  if (!c || !prefill_ms || !decode_ms || !n_steps || max_steps < 0)
    return set_error(FLEX_ERR_INVALID_ARG, "NULL argument or negative capacity");
  *n_steps = 0;
  if (c->ev.empty()) return FLEX_OK;
  const int64_t kept = std::min<int64_t>(c->t_count, FLEX_TIMING_RING);
  const int64_t n = std::min<int64_t>(kept, max_steps);
  for (int64_t k = 0; k < n; ++k) {
    const int64_t slot = (c->t_count - kept + k) % FLEX_TIMING_RING;
    float* dst[2] = {prefill_ms + k, decode_ms + k};
    for (int ph = 0; ph < 2; ++ph) {
      *dst[ph] = 0.f;
      if (!c->has[slot * 2 + ph]) continue;
      hipError_t e = hipEventSynchronize(c->ev[slot * 4 + 2 * ph + 1]);
      if (e != hipSuccess) return hip_fail(e, "timing wait");
      if ((e = hipEventElapsedTime(dst[ph], c->ev[slot * 4 + 2 * ph], c->ev[slot * 4 + 2 * ph + 1])) != hipSuccess)
        return hip_fail(e, "timing read");
    }
  }
  *n_steps = int32_t(n);
  return FLEX_OK;
}

extern "C" int flex_attn_debug_gather(const flex_attn_plan_t* plan, const flex_attn_args* a, int32_t seq,
                                      int32_t seq_len, void* k_out, void* v_out, void* stream) {
  clear_error();
  if (!plan || !a || !a->k_cache || !a->block_table || !k_out)
    return set_error(FLEX_ERR_INVALID_ARG, "NULL argument");
  const flex_attn_shape& sh = plan->shape;
  if (seq < 0 || seq >= plan->info.num_seqs) return set_error(FLEX_ERR_INVALID_ARG, "seq out of range");
  if (seq_len < 0) return set_error(FLEX_ERR_INVALID_ARG, "seq_len < 0");
  const bool has_v = !sh.v_aliases_k;
  if (has_v && (!a->v_cache || !v_out)) return set_error(FLEX_ERR_INVALID_ARG, "v_cache or v_out is NULL");
  const CacheRef kc{static_cast<const uint16_t*>(a->k_cache), a->k_stride[0], a->k_stride[1], a->k_stride[2]};
  const CacheRef vc{static_cast<const uint16_t*>(has_v ? a->v_cache : a->k_cache), a->v_stride[0], a->v_stride[1],
                    a->v_stride[2]};
  const hipError_t e = launch_gather(kc, vc, has_v, a->block_table + int64_t(seq) * a->block_table_stride, seq_len,
                                     sh.page_size, sh.num_kv_heads, sh.head_dim_qk, sh.head_dim_v,
                                     static_cast<uint16_t*>(k_out), static_cast<uint16_t*>(v_out),
                                     static_cast<hipStream_t>(stream));
  return e == hipSuccess ? FLEX_OK : hip_fail(e, "gather launch");
}

extern "C" int flex_attn_workspace_init(void* workspace, size_t bytes, void* stream) {
  clear_error();
  if (bytes == 0) return FLEX_OK;
  if (!workspace || !aligned16(workspace) || bytes % 4)
    return set_error(FLEX_ERR_INVALID_ARG, "workspace must be non-NULL, 16-byte aligned, whole 4-byte words");
  const hipError_t e = launch_fill_zero(workspace, bytes, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? FLEX_OK : hip_fail(e, "fill launch");
}

extern "C" int flex_attn_kv_append(const flex_attn_shape* shape, const flex_attn_append_args* a, void* stream) {
  clear_error();
  if (!shape || !a) return set_error(FLEX_ERR_INVALID_ARG, "shape or args is NULL");
  if (const int st = check_shape(*shape); st != FLEX_OK) return st;
  if (a->n_tokens < 0) return set_error(FLEX_ERR_INVALID_ARG, "n_tokens < 0");
  if (a->n_tokens == 0) return FLEX_OK;
  const bool has_v = !shape->v_aliases_k;
  if (!a->k_new || !a->slot_mapping || !a->k_cache || (has_v && (!a->v_new || !a->v_cache)))
    return set_error(FLEX_ERR_INVALID_ARG, "a required pointer is NULL");
  if (!aligned16(a->k_new) || !aligned16(a->k_cache) || (has_v && (!aligned16(a->v_new) || !aligned16(a->v_cache))))
    return set_error(FLEX_ERR_INVALID_ARG, "new rows and caches must be 16-byte aligned");
  const int64_t Hkv = shape->num_kv_heads, dk = shape->head_dim_qk, dv = shape->head_dim_v;
  if (a->k_new_stride < Hkv * dk || (a->k_new_stride * 2) % 16 ||
      (has_v && (a->v_new_stride < Hkv * dv || (a->v_new_stride * 2) % 16)))
    return set_error(FLEX_ERR_INVALID_ARG, "new-row strides must cover Hkv * d and be 16-byte multiples");
  for (int i = 0; i < 3; ++i) {
    if (a->k_stride[i] <= 0 || (a->k_stride[i] * 2) % 16 || (has_v && (a->v_stride[i] <= 0 || (a->v_stride[i] * 2) % 16)))
      return set_error(FLEX_ERR_INVALID_ARG, "cache strides must be positive multiples of 16 bytes");
  }
  if (a->k_stride[2] < dk || (has_v && a->v_stride[2] < dv))
    return set_error(FLEX_ERR_INVALID_ARG, "cache head stride smaller than the head dimension");
  if (a->num_pages <= 0) return set_error(FLEX_ERR_INVALID_ARG, "num_pages must be positive");
  AppendParams p{};
  p.k_new = static_cast<const uint16_t*>(a->k_new);
  p.v_new = static_cast<const uint16_t*>(has_v ? a->v_new : a->k_new);
  p.k_new_stride = a->k_new_stride;
  p.v_new_stride = has_v ? a->v_new_stride : a->k_new_stride;
  p.slot_mapping = a->slot_mapping;
  p.n_tokens = a->n_tokens;
  p.kc = CacheRef{static_cast<const uint16_t*>(a->k_cache), a->k_stride[0], a->k_stride[1], a->k_stride[2]};
  p.vc = has_v ? CacheRef{static_cast<const uint16_t*>(a->v_cache), a->v_stride[0], a->v_stride[1], a->v_stride[2]}
               : p.kc;
  p.num_slots = a->num_pages * shape->page_size;
  p.P = shape->page_size;
  p.dk = int32_t(dk);
  p.dv = int32_t(dv);
  p.ck = Hkv * dk / 8;
  p.cv = has_v ? Hkv * dv / 8 : 0;
  p.bad_count = a->bad_count;
  const hipError_t e = launch_kv_append(p, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? FLEX_OK : hip_fail(e, "kv append launch");
}
