// Online co-location controller: the step-by-step prefill/decode balance of
// Sec. 3.4 ("Phase-Aware Dispatch", "Avoiding Static PD Imbalance") driven by
// a continuously updated per-phase profile (Sec. 3.3). Host-only, no HIP
// call; the decision rule is restated in include/flexattn.h.
//
// State: for every candidate co-run split k (decode on k * granule CUs,
// prefill on the rest) the decode rate (GB/s) and prefill rate (TFLOP/s)
// observed in that split, the two rates of serial execution, and the ratio
// of one-launch (fused) step times to the serial prediction. Estimates start
// from a prior and move by exponential weighting toward each observed step;
// the first observation of an entry replaces its prior.
#include <algorithm>
#include <cmath>
#include <new>
#include <vector>

#include "host_common.h"

struct flex_ctl {
  flex_ctl_opts o;
  int32_t K;                     // cus_total / granule; index K = serial
  std::vector<double> dec, pre;  // [K + 1], index 0 unused
  std::vector<int64_t> n_dec, n_pre;
  double fused_ratio = 0.0;      // fused step time / serial prediction
  int64_t n_fused = 0;
  double serial_ratio = 1.0;     // serial step time / serial prediction
  int64_t n_serial_steps = 0;
  double last_decode_gbps = 0.0;
  int64_t decisions = 0;
};

namespace {

using flexattn::set_error;

// Alone-rate curve of a profile: linear between points, proportional below
// the first point, flat past the last.
double interp(const std::vector<int32_t>& x, const std::vector<double>& y, double c) {
  if (c <= x.front()) return y.front() * c / x.front();
  for (size_t i = 1; i < x.size(); ++i) {
    if (c <= x[i]) {
      const double t = (c - x[i - 1]) / double(x[i] - x[i - 1]);
      return y[i - 1] + t * (y[i] - y[i - 1]);
    }
  }
  return y.back();
}

void reset_counts(flex_ctl* c) {
  std::fill(c->n_dec.begin(), c->n_dec.end(), 0);
  std::fill(c->n_pre.begin(), c->n_pre.end(), 0);
  c->fused_ratio = c->o.fused_prior;
  c->n_fused = 0;
  c->serial_ratio = 1.0;
  c->n_serial_steps = 0;
  c->last_decode_gbps = 0.0;
}

void seed_prior(flex_ctl* c) {
  const flex_ctl_opts& o = c->o;
  for (int32_t k = 1; k <= c->K; ++k) {
    const double cd = k < c->K ? double(k) * o.granule : double(o.cus_total);
    const double cp = k < c->K ? double(o.cus_total) - cd : double(o.cus_total);
    c->dec[k] = std::min(o.hbm_gbps, cd * o.decode_gbps_per_cu);
    c->pre[k] = cp * o.prefill_tflops_per_cu;
  }
  reset_counts(c);
}

void ewma(double& r, int64_t& n, double obs, double alpha) {
  r = n == 0 ? obs : (1.0 - alpha) * r + alpha * obs;
  ++n;
}

}  // namespace

extern "C" int flex_ctl_create(const flex_ctl_opts* opts, flex_ctl_t** out) {
  flexattn::clear_error();
  if (!out) return set_error(FLEX_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  flex_ctl_opts o{};
  if (opts) o = *opts;
  if (!o.cus_total) o.cus_total = 256;
  if (!o.granule) o.granule = 64;
  if (!o.explore_every) o.explore_every = 16;
  if (!o.backlog_seqs) o.backlog_seqs = 256;
  if (!o.backlog_prefill_tokens) o.backlog_prefill_tokens = 8192;
  if (o.alpha == 0.0) o.alpha = 0.25;
  if (o.tolerance == 0.0) o.tolerance = 0.03;
  if (o.sat_frac == 0.0) o.sat_frac = 0.6;
  if (o.hbm_gbps == 0.0) o.hbm_gbps = 8000.0;
  if (o.corun_overhead_us == 0.0) o.corun_overhead_us = 10.0;
  if (o.decode_gbps_per_cu == 0.0) o.decode_gbps_per_cu = 60.0;
  if (o.prefill_tflops_per_cu == 0.0) o.prefill_tflops_per_cu = 5.0;
  if (o.fused_prior == 0.0) o.fused_prior = 0.9;
  if (o.cus_total < 2 || o.granule < 1 || o.cus_total % o.granule || o.cus_total / o.granule < 2)
    return set_error(FLEX_ERR_INVALID_ARG, "granule must divide cus_total into at least two parts");
  if (!(o.alpha > 0.0 && o.alpha <= 1.0) || !(o.tolerance >= 0.0) || !(o.sat_frac > 0.0) ||
      !(o.hbm_gbps > 0.0) || !(o.corun_overhead_us >= 0.0) || !(o.decode_gbps_per_cu > 0.0) ||
      !(o.prefill_tflops_per_cu > 0.0) || !(o.fused_prior > 0.0) || o.backlog_seqs < 0 ||
      o.backlog_prefill_tokens < 0)
    return set_error(FLEX_ERR_INVALID_ARG, "controller options out of range");
  flex_ctl* c = new (std::nothrow) flex_ctl();
  if (!c) return set_error(FLEX_ERR_INTERNAL, "out of host memory");
  c->o = o;
  c->K = o.cus_total / o.granule;
  c->dec.assign(c->K + 1, 0.0);
  c->pre.assign(c->K + 1, 0.0);
  c->n_dec.assign(c->K + 1, 0);
  c->n_pre.assign(c->K + 1, 0);
  seed_prior(c);
  *out = c;
  return FLEX_OK;
}

extern "C" void flex_ctl_destroy(flex_ctl_t* ctl) { delete ctl; }

extern "C" int flex_ctl_set_profile(flex_ctl_t* c, int32_t n, const int32_t* cus, const double* dg,
                                    const double* pt) {
  flexattn::clear_error();
  if (!c || n < 1 || !cus || !dg || !pt) return set_error(FLEX_ERR_INVALID_ARG, "NULL argument or n < 1");
  std::vector<int32_t> x(cus, cus + n);
  std::vector<double> d(dg, dg + n), p(pt, pt + n);
  for (int32_t i = 0; i < n; ++i) {
    if (x[i] <= 0 || (i && x[i] <= x[i - 1]) || !(d[i] > 0.0) || !(p[i] > 0.0))
      return set_error(FLEX_ERR_INVALID_ARG, "profile CU counts must ascend and rates be positive");
  }
  for (int32_t k = 1; k <= c->K; ++k) {
    const double cd = k < c->K ? double(k) * c->o.granule : double(c->o.cus_total);
    const double cp = k < c->K ? double(c->o.cus_total) - cd : double(c->o.cus_total);
    c->dec[k] = interp(x, d, cd);
    c->pre[k] = interp(x, p, cp);
  }
  reset_counts(c);
  return FLEX_OK;
}

extern "C" int flex_ctl_observe(flex_ctl_t* c, const flex_ctl_observation* ob) {
  flexattn::clear_error();
  if (!c || !ob) return set_error(FLEX_ERR_INVALID_ARG, "NULL argument");
  // the serial prediction for the same work, from the current estimates (us)
  const double pred = (ob->decode_bytes > 0.0 ? ob->decode_bytes / (c->dec[c->K] * 1e3) : 0.0) +
                      (ob->prefill_flops > 0.0 ? ob->prefill_flops / (c->pre[c->K] * 1e6) : 0.0);
  if (ob->fused) {
    if (ob->step_ms > 0.0 && pred > 0.0) ewma(c->fused_ratio, c->n_fused, ob->step_ms * 1e3 / pred, c->o.alpha);
    return FLEX_OK;
  }
  int32_t k;
  if (ob->cus_decode == 0 || ob->cus_decode == c->o.cus_total) {
    k = c->K;
  } else {
    if (ob->cus_decode < 0 || ob->cus_decode % c->o.granule || ob->cus_decode > c->o.cus_total)
      return set_error(FLEX_ERR_INVALID_ARG, "cus_decode is not a candidate split");
    k = ob->cus_decode / c->o.granule;
  }
  if (k == c->K && ob->step_ms > 0.0 && pred > 0.0)
    ewma(c->serial_ratio, c->n_serial_steps, ob->step_ms * 1e3 / pred, c->o.alpha);
  if (ob->decode_ms > 0.0 && ob->decode_bytes > 0.0) {
    const double r = ob->decode_bytes / (ob->decode_ms * 1e-3) / 1e9;
    ewma(c->dec[k], c->n_dec[k], r, c->o.alpha);
    c->last_decode_gbps = r;
  }
  if (ob->prefill_ms > 0.0 && ob->prefill_flops > 0.0) {
    const double r = ob->prefill_flops / (ob->prefill_ms * 1e-3) / 1e12;
    ewma(c->pre[k], c->n_pre[k], r, c->o.alpha);
  }
  return FLEX_OK;
}

extern "C" int flex_ctl_decide(flex_ctl_t* c, const flex_ctl_signals* sg, flex_ctl_decision* out) {
  flexattn::clear_error();
  if (!c || !sg || !out) return set_error(FLEX_ERR_INVALID_ARG, "NULL argument");
  const flex_ctl_opts& o = c->o;
  const int32_t K = c->K;
  ++c->decisions;
  const double B = sg->decode_bytes, F = sg->prefill_flops;
  // predicted phase times in microseconds
  auto t_dec = [&](int32_t k) { return B > 0.0 ? B / (c->dec[k] * 1e3) : 0.0; };
  auto t_pre = [&](int32_t k) { return F > 0.0 ? F / (c->pre[k] * 1e6) : 0.0; };
  auto serial = [&](int32_t reason) {
    out->mode = FLEX_MODE_SERIAL;
    out->cus_decode = o.cus_total;
    out->cus_prefill = o.cus_total;
    out->reason = reason;
    out->predicted_us = t_dec(K) + t_pre(K);
    return FLEX_OK;
  };
  if (!(B > 0.0) || !(F > 0.0) || sg->active_decode_seqs == 0) return serial(FLEX_CTL_ONE_PHASE);

  std::vector<double> T(K + 1, 0.0);
  int32_t best = 1;
  for (int32_t k = 1; k <= K; ++k) {
    if (k == K) T[k] = t_dec(k) + t_pre(k);
    else if (sg->decode_tail && t_pre(k) >= flexattn::kTailMinPrefillUs && t_dec(k) > t_pre(k))
      // decode's rest, at the all-CU rate, after the prefill
      T[k] = t_pre(k) + (B - c->dec[k] * 1e3 * t_pre(k)) / (c->dec[K] * 1e3) + o.corun_overhead_us;
    else T[k] = std::max(t_dec(k), t_pre(k)) + o.corun_overhead_us;
    if (T[k] < T[best]) best = k;
  }
  // One-launch form: the serial prediction times the ratio of observed fused
  // to observed serial step times (both against the serial prediction).
  const bool has_fused = sg->fused_available != 0;
  const double Tf = has_fused ? c->fused_ratio / c->serial_ratio * T[K] : 0.0;
  const bool explore_turn = o.explore_every > 0 && c->decisions % o.explore_every == 0;
  const bool fused_turn = explore_turn && has_fused && (c->decisions / o.explore_every) % 4 == 3;
  auto fused = [&](int32_t reason) {
    out->mode = FLEX_MODE_FUSED;
    out->cus_decode = o.cus_total;
    out->cus_prefill = o.cus_total;
    out->reason = reason;
    out->predicted_us = Tf;
    return FLEX_OK;
  };
  if (best == K) {
    if (has_fused && Tf < T[K]) return fused(FLEX_CTL_FUSED_FASTER);
    if (fused_turn) return fused(FLEX_CTL_EXPLORE);
    return serial(FLEX_CTL_SERIAL_FASTER);
  }

  int32_t lo = best, hi = best;   // co-run splits within the band
  for (int32_t k = 1; k < K; ++k) {
    if (T[k] <= T[best] * (1.0 + o.tolerance)) {
      lo = std::min(lo, k);
      hi = std::max(hi, k);
    }
  }
  int32_t choice = best, reason = FLEX_CTL_BEST;
  if (sg->pending_decode_seqs >= o.backlog_seqs) {
    choice = hi;
    reason = FLEX_CTL_BACKLOG;
  } else if (c->last_decode_gbps >= o.sat_frac * o.hbm_gbps) {
    choice = lo;
    reason = FLEX_CTL_BW_SATURATED;
  } else if (sg->pending_prefill_tokens >= o.backlog_prefill_tokens) {
    choice = lo;
    reason = FLEX_CTL_PREFILL_BACKLOG;
  }
  const bool fused_best = has_fused && Tf < T[best];
  if (fused_turn && !fused_best) return fused(FLEX_CTL_EXPLORE);
  if (fused_best) return fused(FLEX_CTL_FUSED_FASTER);
  if (explore_turn) {
    const int32_t step = (c->decisions / o.explore_every) % 2 ? 1 : -1;
    int32_t k = choice + step;
    if (k < 1 || k >= K) k = choice - step;
    if (k >= 1 && k < K) {
      choice = k;
      reason = FLEX_CTL_EXPLORE;
    }
  }
  out->mode = FLEX_MODE_CORUN;
  out->cus_decode = choice * o.granule;
  out->cus_prefill = o.cus_total - out->cus_decode;
  out->reason = reason;
  out->predicted_us = T[choice];
  return FLEX_OK;
}

extern "C" int flex_ctl_estimates(const flex_ctl_t* c, double* dg, double* pt, int32_t capacity) {
  flexattn::clear_error();
  if (!c || !dg || !pt) return set_error(FLEX_ERR_INVALID_ARG, "NULL argument");
  if (capacity < c->K) return set_error(FLEX_ERR_INVALID_ARG, "capacity below cus_total / granule");
  for (int32_t k = 1; k <= c->K; ++k) {
    dg[k - 1] = c->dec[k];
    pt[k - 1] = c->pre[k];
  }
  return FLEX_OK;
}

// ---------------------------------------------------------------------------
// Time-slice scheduler (temporal multiplexing, Sec. 3 and Sec. 3.4; the
// time-slice ratio of Sec. 4): one phase per step on the whole device, the
// phase chosen so that decode's share of the windowed device time tracks
// decode_share. A deficit rule: whichever phase is below its share runs next.

struct flex_ts {
  double share;
  double decay;
  double t_dec = 0.0;
  double t_pre = 0.0;
};

extern "C" int flex_ts_create(const flex_ts_opts* opts, flex_ts_t** out) {
  flexattn::clear_error();
  if (!out) return set_error(FLEX_ERR_INVALID_ARG, "NULL argument");
  *out = nullptr;
  flex_ts_opts o{};
  if (opts) o = *opts;
  if (o.decode_share == 0.0) o.decode_share = 0.5;
  if (o.decay == 0.0) o.decay = 1.0;
  if (!(o.decode_share > 0.0 && o.decode_share < 1.0))
    return set_error(FLEX_ERR_INVALID_ARG, "decode_share must lie in (0, 1)");
  if (!(o.decay > 0.0 && o.decay <= 1.0)) return set_error(FLEX_ERR_INVALID_ARG, "decay must lie in (0, 1]");
  flex_ts* t = new (std::nothrow) flex_ts;
  if (!t) return set_error(FLEX_ERR_INTERNAL, "out of host memory");
  t->share = o.decode_share;
  t->decay = o.decay;
  *out = t;
  return FLEX_OK;
}

extern "C" void flex_ts_destroy(flex_ts_t* t) { delete t; }

extern "C" int flex_ts_next(const flex_ts_t* t, int32_t decode_ready, int32_t prefill_ready, int32_t* phase) {
  flexattn::clear_error();
  if (!t || !phase) return set_error(FLEX_ERR_INVALID_ARG, "NULL argument");
  if (!decode_ready && !prefill_ready) return set_error(FLEX_ERR_INVALID_ARG, "neither phase has work");
  if (!prefill_ready) *phase = FLEX_TS_DECODE;
  else if (!decode_ready) *phase = FLEX_TS_PREFILL;
  else *phase = t->t_dec * (1.0 - t->share) <= t->t_pre * t->share ? FLEX_TS_DECODE : FLEX_TS_PREFILL;
  return FLEX_OK;
}

extern "C" int flex_ts_observe(flex_ts_t* t, int32_t phase, double ms) {
  flexattn::clear_error();
  if (!t) return set_error(FLEX_ERR_INVALID_ARG, "NULL argument");
  if (phase != FLEX_TS_DECODE && phase != FLEX_TS_PREFILL) return set_error(FLEX_ERR_INVALID_ARG, "unknown phase");
  if (!(ms >= 0.0) || !std::isfinite(ms)) return set_error(FLEX_ERR_INVALID_ARG, "duration must be finite and >= 0");
  t->t_dec *= t->decay;
  t->t_pre *= t->decay;
  (phase == FLEX_TS_DECODE ? t->t_dec : t->t_pre) += ms;
  return FLEX_OK;
}

extern "C" int flex_ts_totals(const flex_ts_t* t, double* decode_ms, double* prefill_ms) {
  flexattn::clear_error();
  if (!t || !decode_ms || !prefill_ms) return set_error(FLEX_ERR_INVALID_ARG, "NULL argument");
  *decode_ms = t->t_dec;
  *prefill_ms = t->t_pre;
  return FLEX_OK;
}
