// Host-side fuzz driver for the planner and the co-location controller, built
// with the address and undefined-behaviour sanitizers by tests/test_host_sanitized.py.
// Feeds random (valid and invalid) batch metadata and options to
// flex_attn_plan, exports every plan, and drives a controller through random
// observe/decide sequences. Any sanitizer report aborts the process.
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "flexattn.h"

int main(int argc, char** argv) {
  const int iters = argc > 1 ? std::atoi(argv[1]) : 2000;
  std::mt19937 rng(12345);
  auto pick = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  const flex_attn_shape shapes[] = {
      {28, 4, 128, 128, 16, 0.088f, 0}, {4, 1, 64, 64, 16, 0.125f, 0},   {32, 2, 128, 128, 64, 0.1f, 0},
      {128, 1, 576, 512, 64, 0.072f, 1}, {64, 1, 576, 512, 64, 0.07f, 1}, {16, 16, 192, 128, 64, 0.07f, 0},
      {30, 4, 128, 128, 16, 0.1f, 0},    {28, 4, 96, 96, 16, 0.1f, 0},    {28, 4, 128, 128, 32, 0.1f, 0}};
  int ok = 0, rejected = 0;
  for (int it = 0; it < iters; ++it) {
    const flex_attn_shape sh = shapes[pick(0, int(sizeof(shapes) / sizeof(shapes[0])) - 1)];
    const int B = pick(0, 40);
    std::vector<int32_t> qsl(B + 1, 0), ls(B);
    for (int s = 0; s < B; ++s) {
      const int L = pick(0, 5000);
      int n = pick(0, 4) == 0 ? L : pick(0, 3) == 0 ? 0 : 1;
      if (pick(0, 50) == 0) n = L + 1;             // invalid: more new tokens than keys
      ls[s] = L;
      qsl[s + 1] = qsl[s] + n;
    }
    if (B && pick(0, 60) == 0) qsl[1] = -1;        // invalid: decreasing
    int maxp = 1;
    for (int L : ls) maxp = std::max(maxp, (L + sh.page_size - 1) / sh.page_size);
    if (pick(0, 40) == 0) maxp = 0;                // invalid: too small
    flex_attn_plan_opts o{};
    o.cus_decode = pick(0, 3) == 0 ? -1 : pick(0, 1) ? 0 : 32 * pick(1, 7);
    o.bm = pick(0, 2) == 0 ? 16 * pick(0, 8) : 0;
    o.min_split_tokens = pick(0, 1) ? 0 : pick(1, 4096);
    o.wg_per_cu = pick(0, 1) ? 0 : pick(1, 8);
    o.cus_total = pick(0, 1) ? 0 : pick(1, 512);
    flex_attn_plan_t* plan = nullptr;
    const int st = flex_attn_plan(&sh, pick(0, 5) ? &o : nullptr, B, qsl.data(), ls.data(), maxp, &plan);
    if (st != FLEX_OK) {
      ++rejected;
      continue;
    }
    ++ok;
    flex_attn_plan_info info;
    if (flex_attn_plan_info_get(plan, &info) != FLEX_OK) return 2;
    std::vector<int32_t> words(info.plan_words);
    if (flex_attn_plan_export(plan, words.data(), words.size()) != FLEX_OK) return 3;
    flex_attn_plan_destroy(plan);
  }
  // controller
  for (int rep = 0; rep < 50; ++rep) {
    flex_ctl_opts co{};
    co.granule = 32 << pick(0, 2);
    co.explore_every = pick(-1, 9);
    flex_ctl_t* ctl = nullptr;
    if (flex_ctl_create(&co, &ctl) != FLEX_OK) return 4;
    if (pick(0, 1)) {
      const int32_t cus[] = {32, 64, 128, 256};
      const double dg[] = {1500, 2800, 4700, 5600}, pt[] = {130, 270, 500, 750};
      if (flex_ctl_set_profile(ctl, 4, cus, dg, pt) != FLEX_OK) return 5;
    }
    for (int s = 0; s < 200; ++s) {
      flex_ctl_signals sg{double(pick(0, 3000)) * 1e6, double(pick(0, 3000)) * 1e9, pick(0, 20000), pick(0, 500),
                          pick(0, 300), pick(0, 1)};
      flex_ctl_decision d;
      if (flex_ctl_decide(ctl, &sg, &d) != FLEX_OK) return 6;
      flex_ctl_observation ob{d.mode == FLEX_MODE_CORUN ? d.cus_decode : 0, sg.decode_bytes, sg.prefill_flops,
                              pick(0, 1000) * 1e-3, pick(0, 5000) * 1e-3,
                              d.mode == FLEX_MODE_FUSED ? 1 : 0, pick(0, 5000) * 1e-3};
      if (flex_ctl_observe(ctl, &ob) != FLEX_OK) return 7;
    }
    double dg[64], pt[64];
    if (flex_ctl_estimates(ctl, dg, pt, 64) != FLEX_OK) return 8;
    flex_ctl_destroy(ctl);
  }
  // time-slice scheduler: random targets, windows, readiness and durations
  for (int it = 0; it < iters / 10 + 1; ++it) {
    flex_ts_opts to{std::uniform_real_distribution<double>(0.01, 0.99)(rng), pick(0, 1) ? 1.0 : 0.9};
    flex_ts_t* ts = nullptr;
    if (flex_ts_create(&to, &ts) != FLEX_OK) return 10;
    for (int s = 0; s < 50; ++s) {
      const int dr = pick(0, 1), pr = pick(0, 1);
      int32_t ph = -1;
      const int st = flex_ts_next(ts, dr, pr, &ph);
      if (!dr && !pr) {
        if (st != FLEX_ERR_INVALID_ARG) return 11;
        continue;
      }
      if (st != FLEX_OK || (ph == FLEX_TS_DECODE ? !dr : !pr)) return 12;
      if (flex_ts_observe(ts, ph, pick(0, 1000) * 1e-3) != FLEX_OK) return 13;
    }
    double d = -1, p = -1;
    if (flex_ts_totals(ts, &d, &p) != FLEX_OK || d < 0 || p < 0) return 14;
    flex_ts_destroy(ts);
  }
  std::printf("plans ok %d rejected %d\n", ok, rejected);
  return ok > 0 && rejected > 0 ? 0 : 9;
}
