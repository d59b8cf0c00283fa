"""Re-derivations of the host policies: the online co-location controller's
decisions and, at the end of the module, the time-slice scheduler's phase
choices (``TimeSlice``).

TEST INFRASTRUCTURE. Only ``tests/`` may import this module. The library never
does, and this module imports nothing from the library.

The paper's runtime rebalances prefill and decode step by step from five
signals (Sec. 3.4, "Phase-Aware Dispatch"): pending work of each phase,
recent per-phase execution times, memory-bandwidth pressure, decode progress
and active sequences, device utilisation; decode near bandwidth saturation
cedes compute to prefill, a decode backlog takes more. Its profile is coarse
and updated while serving (Sec. 3.3). The paper gives no formula, so the
library fixes one (stated in include/flexattn.h) and this module restates it
independently, step by step, so that tests can compare every decision of the
library with it exactly:

* candidates: co-run with decode on k * g CUs (k = 1 .. K-1, K = cus_total / g)
  and serial (index K);
* estimates per candidate: decode GB/s and prefill TFLOP/s, seeded by a prior
  (min(hbm, cus * bw_cu), cus * tflops_cu) or by a profile (linear
  interpolation of alone rates, proportional below the first point, flat past
  the last), then exponentially weighted toward each observation (the first
  observation replaces the prior);
* prediction in microseconds: co-run max(B / (dec * 1e3), F / (pre * 1e6)) +
  overhead, serial B / (dec * 1e3) + F / (pre * 1e6);
* choice: serial if a phase is empty or serial predicts strictly fastest (ties
  go to the smaller index); else, among co-run splits within
  (1 + tolerance) of the best, the largest decode share under a decode backlog,
  else the smallest under bandwidth pressure (last observed decode rate >=
  sat_frac * hbm) or a prefill backlog, else the best; every explore_every-th
  decision moves to a neighbour (+1 on odd multiples, -1 on even ones, the
  other way at the ends);
* one-launch (fused) form, when the step has one: predicted as the serial
  prediction times fused_ratio / serial_ratio, two running ratios of whole
  step times to the serial prediction from the current serial estimates
  (before the observation updates them): fused steps feed fused_ratio (prior
  fused_prior), serial steps that report their step time feed serial_ratio
  (prior 1), each first observation replacing the prior; a profile resets
  both. It is chosen
  when its prediction is strictly below serial's (if serial beats every
  co-run split) or the best co-run split's (otherwise). On an explore turn
  whose index (decisions // explore_every) is 3 mod 4, a step that has the
  form and did not choose it runs it instead (reason EXPLORE), before any
  neighbour move; a serial choice makes no neighbour move.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

ONE_PHASE, BEST, SERIAL_FASTER, BACKLOG, BW_SATURATED, EXPLORE, PREFILL_BACKLOG, FUSED_FASTER = range(8)
MODE_SERIAL, MODE_CORUN, MODE_FUSED = 0, 1, 2


@dataclass
class CtlOpts:
    cus_total: int = 256
    granule: int = 64
    explore_every: int = 16
    backlog_seqs: int = 256
    backlog_prefill_tokens: int = 8192
    alpha: float = 0.25
    tolerance: float = 0.03
    sat_frac: float = 0.6
    hbm_gbps: float = 8000.0
    corun_overhead_us: float = 10.0
    decode_gbps_per_cu: float = 60.0
    prefill_tflops_per_cu: float = 5.0
    fused_prior: float = 0.9


OC_DEFAULTS = CtlOpts()


@dataclass
class Controller:
    o: CtlOpts
    dec: List[float] = field(default_factory=list)
    pre: List[float] = field(default_factory=list)
    n_dec: List[int] = field(default_factory=list)
    n_pre: List[int] = field(default_factory=list)
    last_bw: float = 0.0
    decisions: int = 0
    fused_ratio: float = 0.0
    n_fused: int = 0
    serial_ratio: float = 1.0
    n_serial_steps: int = 0

    @property
    def K(self) -> int:
        return self.o.cus_total // self.o.granule

    def shares(self, k: int):
        """(decode CUs, prefill CUs) of candidate k (K = serial: both get all)."""
        if k == self.K:
            return float(self.o.cus_total), float(self.o.cus_total)
        cd = float(k * self.o.granule)
        return cd, float(self.o.cus_total) - cd

    def __post_init__(self):
        # a zero option takes its default, as in the library's options
        d = OC_DEFAULTS
        for name in vars(d):
            if getattr(self.o, name) == 0:
                setattr(self.o, name, getattr(d, name))
        K = self.K
        self.dec = [0.0] * (K + 1)
        self.pre = [0.0] * (K + 1)
        for k in range(1, K + 1):
            cd, cp = self.shares(k)
            self.dec[k] = min(self.o.hbm_gbps, cd * self.o.decode_gbps_per_cu)
            self.pre[k] = cp * self.o.prefill_tflops_per_cu
        self.n_dec = [0] * (K + 1)
        self.n_pre = [0] * (K + 1)
        self.fused_ratio, self.n_fused = self.o.fused_prior, 0
        self.serial_ratio, self.n_serial_steps = 1.0, 0

    def set_profile(self, cus: Sequence[int], dgbps: Sequence[float], ptflops: Sequence[float]):
        def curve(ys, c):
            if c <= cus[0]:
                return ys[0] * c / cus[0]
            for i in range(1, len(cus)):
                if c <= cus[i]:
                    t = (c - cus[i - 1]) / float(cus[i] - cus[i - 1])
                    return ys[i - 1] + t * (ys[i] - ys[i - 1])
            return ys[-1]
        for k in range(1, self.K + 1):
            cd, cp = self.shares(k)
            self.dec[k] = curve(dgbps, cd)
            self.pre[k] = curve(ptflops, cp)
        self.n_dec = [0] * (self.K + 1)
        self.n_pre = [0] * (self.K + 1)
        self.last_bw = 0.0
        self.fused_ratio, self.n_fused = self.o.fused_prior, 0
        self.serial_ratio, self.n_serial_steps = 1.0, 0

    def _blend(self, table, counts, k, value):
        table[k] = value if counts[k] == 0 else (1.0 - self.o.alpha) * table[k] + self.o.alpha * value
        counts[k] += 1

    def serial_prediction_us(self, B: float, F: float) -> float:
        K = self.K
        return (B / (self.dec[K] * 1e3) if B > 0 else 0.0) + (F / (self.pre[K] * 1e6) if F > 0 else 0.0)

    def observe(self, cus_decode: int, decode_bytes: float, prefill_flops: float,
                decode_ms: float, prefill_ms: float, fused: bool = False, step_ms: float = 0.0):
        base = self.serial_prediction_us(decode_bytes, prefill_flops)
        if fused:
            if step_ms > 0 and base > 0:
                r = step_ms * 1e3 / base
                self.fused_ratio = r if self.n_fused == 0 else (1.0 - self.o.alpha) * self.fused_ratio + self.o.alpha * r
                self.n_fused += 1
            return
        k = self.K if cus_decode in (0, self.o.cus_total) else cus_decode // self.o.granule
        if k == self.K and step_ms > 0 and base > 0:
            r = step_ms * 1e3 / base
            self.serial_ratio = r if self.n_serial_steps == 0 else \
                (1.0 - self.o.alpha) * self.serial_ratio + self.o.alpha * r
            self.n_serial_steps += 1
        if decode_ms > 0 and decode_bytes > 0:
            r = decode_bytes / (decode_ms * 1e-3) / 1e9
            self._blend(self.dec, self.n_dec, k, r)
            self.last_bw = r
        if prefill_ms > 0 and prefill_flops > 0:
            self._blend(self.pre, self.n_pre, k, prefill_flops / (prefill_ms * 1e-3) / 1e12)

    def decide(self, decode_bytes: float, prefill_flops: float, pending_prefill_tokens: int = 0,
               pending_decode_seqs: int = 0, active_decode_seqs: int = 1, fused_available: bool = False,
               decode_tail: bool = False) -> dict:
        o, K = self.o, self.K
        self.decisions += 1
        B, F = decode_bytes, prefill_flops

        def phase_times(k):
            td = B / (self.dec[k] * 1e3) if B > 0 else 0.0
            tp = F / (self.pre[k] * 1e6) if F > 0 else 0.0
            return td, tp

        def serial(reason):
            td, tp = phase_times(K)
            return dict(mode=MODE_SERIAL, cus_decode=o.cus_total, cus_prefill=o.cus_total,
                        reason=reason, predicted_us=td + tp)

        if not (B > 0) or not (F > 0) or active_decode_seqs == 0:
            return serial(ONE_PHASE)
        pred = {}
        for k in range(1, K + 1):
            td, tp = phase_times(k)
            if k == K:
                pred[k] = td + tp
            elif decode_tail and tp >= 100.0 and td > tp:   # (the plan's tail needs a 100 us prefill)
                # the co-run decode share streams until the prefill ends; the
                # rest runs on every CU at the rate decode reaches there
                bytes_left = B - self.dec[k] * 1e3 * tp
                pred[k] = tp + bytes_left / (self.dec[K] * 1e3) + o.corun_overhead_us
            else:
                pred[k] = max(td, tp) + o.corun_overhead_us
        best = 1
        for k in range(2, K + 1):
            if pred[k] < pred[best]:
                best = k
        t_fused = self.fused_ratio / self.serial_ratio * pred[K] if fused_available else None
        explore = o.explore_every > 0 and self.decisions % o.explore_every == 0
        explore_fused = explore and fused_available and (self.decisions // o.explore_every) % 4 == 3

        def fused(reason):
            return dict(mode=MODE_FUSED, cus_decode=o.cus_total, cus_prefill=o.cus_total, reason=reason,
                        predicted_us=t_fused)

        if best == K:
            if t_fused is not None and t_fused < pred[K]:
                return fused(FUSED_FASTER)
            if explore_fused:
                return fused(EXPLORE)
            return serial(SERIAL_FASTER)
        band = [k for k in range(1, K) if pred[k] <= pred[best] * (1.0 + o.tolerance)]
        choice, reason = best, BEST
        if pending_decode_seqs >= o.backlog_seqs:
            choice, reason = max(band), BACKLOG
        elif self.last_bw >= o.sat_frac * o.hbm_gbps:
            choice, reason = min(band), BW_SATURATED
        elif pending_prefill_tokens >= o.backlog_prefill_tokens:
            choice, reason = min(band), PREFILL_BACKLOG
        fused_wins = t_fused is not None and t_fused < pred[best]
        if explore_fused and not fused_wins:
            return fused(EXPLORE)
        if fused_wins:
            return fused(FUSED_FASTER)
        if explore:
            step = 1 if (self.decisions // o.explore_every) % 2 else -1
            k = choice + step
            if not 1 <= k < K:
                k = choice - step
            if 1 <= k < K:
                choice, reason = k, EXPLORE
        return dict(mode=MODE_CORUN, cus_decode=choice * o.granule, cus_prefill=o.cus_total - choice * o.granule,
                    reason=reason, predicted_us=pred[choice])

    def estimates(self):
        return self.dec[1:], self.pre[1:]


# ---------------------------------------------------------------------------
# Time-slice scheduler (temporal multiplexing of the phases; Sec. 3, Sec. 3.4;
# the time-slice ratio of Sec. 4). The paper fixes no rule; the library's is a
# deficit rule, restated here: each step runs one phase on the whole device;
# with both phases ready, decode runs when its share of the windowed device
# time is at most decode_share, i.e. t_dec * (1 - share) <= t_pre * share in
# double precision (ties to decode), else prefill; with one ready, that one.
# Before each observation both totals are multiplied by decay.

TS_DECODE, TS_PREFILL = 0, 1


class TimeSlice:
    def __init__(self, decode_share: float = 0.0, decay: float = 0.0):
        self.share = decode_share if decode_share != 0.0 else 0.5
        self.decay = decay if decay != 0.0 else 1.0
        if not (0.0 < self.share < 1.0) or not (0.0 < self.decay <= 1.0):
            raise ValueError("decode_share in (0, 1), decay in (0, 1]")
        self.t_dec = 0.0
        self.t_pre = 0.0

    def next(self, decode_ready: bool, prefill_ready: bool) -> int:
        if not decode_ready and not prefill_ready:
            raise ValueError("neither phase has work")
        if not prefill_ready:
            return TS_DECODE
        if not decode_ready:
            return TS_PREFILL
        return TS_DECODE if self.t_dec * (1.0 - self.share) <= self.t_pre * self.share else TS_PREFILL

    def observe(self, phase: int, ms: float):
        self.t_dec *= self.decay
        self.t_pre *= self.decay
        if phase == TS_DECODE:
            self.t_dec += ms
        else:
            self.t_pre += ms
