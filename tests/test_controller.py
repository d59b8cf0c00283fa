"""The online co-location controller (host policy, CPU only).

Parity: every decision of the library's controller equals the re-derivation
in oracle/controller.py on long random observe/decide sequences (exact float
equality of the predicted time), one-launch steps included. Pins, independent
of both: the rule's directions from the paper (Sec. 3.4: bandwidth saturation
cedes CUs to prefill, decode backlog takes more), monotonicity in the step's
work, the argmin on a profile whose optimum is known in closed form,
convergence of the estimates, the exploration pattern, the one-launch form's
ratio rule in closed form, and one planted mistake.
"""
import random

import pytest

import oracle.controller as OC
from paper_2606_04415_amd import flexattn as F


def both(**opts):
    return F.Controller(**opts), OC.Controller(OC.CtlOpts(**opts))


def same(a, b):
    assert a["mode"] == b["mode"] and a["cus_decode"] == b["cus_decode"] and a["cus_prefill"] == b["cus_prefill"]
    assert a["reason"] == b["reason"], (a, b)
    assert a["predicted_us"] == b["predicted_us"], (a, b)


@pytest.mark.parametrize("seed", range(6))
def test_decisions_match_the_re_derivation(seed):
    rng = random.Random(seed)
    opts = dict(granule=rng.choice([32, 64, 128]), explore_every=rng.choice([0, -1, 5, 16]),
                backlog_seqs=rng.choice([64, 256]), tolerance=rng.choice([0.0, 1e-12, 0.2]))
    lib, ref = both(**opts)
    if seed % 2:
        prof = ([32, 64, 128, 192, 256], [1500.0, 2800.0, 4660.0, 5600.0, 5550.0], [135.0, 268.0, 488.0, 517.0, 733.0])
        lib.set_profile(*prof)
        ref.set_profile(*prof)
    K = 256 // opts["granule"]
    modes = set()
    for step in range(400):
        B = rng.choice([0.0, rng.uniform(1e8, 3e9)])
        Fl = rng.choice([0.0, rng.uniform(1e10, 3e12)])
        sig = dict(pending_prefill_tokens=rng.randrange(0, 20000), pending_decode_seqs=rng.randrange(0, 400),
                   active_decode_seqs=rng.randrange(0, 300), fused_available=rng.random() < 0.7,
                   decode_tail=rng.random() < 0.5)
        a = lib.decide(B, Fl, **sig)
        b = ref.decide(B, Fl, **sig)
        same(a, b)
        modes.add(a["mode"])
        if a["mode"] == F.FLEX_MODE_FUSED:
            obs = (256, B, Fl, 0.0, 0.0, True, rng.uniform(0.05, 6.0))
        else:
            cd = a["cus_decode"] if a["mode"] == F.FLEX_MODE_CORUN else rng.choice([0, 256])
            obs = (cd, B, Fl, rng.uniform(0.05, 3.0) if B else 0.0, rng.uniform(0.05, 9.0) if Fl else 0.0,
                   False, rng.choice([0.0, rng.uniform(0.05, 6.0)]))
        lib.observe(*obs)
        ref.observe(*obs)
    assert lib.estimates() == ref.estimates()
    assert F.FLEX_MODE_FUSED in modes


def profile_linear(ctl, bw_per_cu, sat_gbps, tf_per_cu):
    """A profile with decode rate min(sat, bw_per_cu * c), prefill tf_per_cu * c."""
    cus = list(range(32, 257, 32))
    ctl.set_profile(cus, [min(sat_gbps, bw_per_cu * c) for c in cus], [tf_per_cu * c for c in cus])


def test_argmin_matches_closed_form_optimum():
    # decode 40 GB/s per CU, saturating at 5120 GB/s from 128 CUs; prefill 4 TFLOP/s
    # per CU. Below saturation the phase times balance where B / (40 c) = F / (4 (256 - c));
    # B, F are chosen so that this happens at c = 96: F = B * 4e12 * 160 / (40 * 96e9).
    # Serial then takes B / 5120 GB/s + F / 1024 TFLOP/s = 358 us, co-run 260 us.
    ctl = F.Controller(granule=32, explore_every=-1, tolerance=1e-12, corun_overhead_us=1e-9)
    profile_linear(ctl, 40.0, 5120.0, 4.0)
    B = 1.0e9
    Fl = B * 4e12 * 160 / (40 * 96e9)
    d = ctl.decide(B, Fl, active_decode_seqs=10)
    assert d["mode"] == F.FLEX_MODE_CORUN and d["cus_decode"] == 96 and d["reason"] == F.FLEX_CTL_BEST
    # at the balance point both phases take B / (40 GB/s * 96) = 260.4 us
    assert abs(d["predicted_us"] - B / (40e9 * 96) * 1e6) < 1e-6


def test_decode_tail_moves_the_best_split():
    # Same linear profile; B = 1.2 GB, F such that the prefill takes 240 us on 160
    # CUs. Slower phase: 96 decode CUs give max(312.5, 240), 128 give max(234.4,
    # 300) = 300 us, the best. With a decode tail, 96 decode CUs stream 0.9216 GB
    # during the prefill's 240 us and the rest 0.2784 GB at 5120 GB/s (54.375 us):
    # 294.375 us, better than 128 (300, decode done first) and 64 (200 + 0.688 GB
    # at 5120 GB/s = 334.4 us).
    ctl = F.Controller(granule=32, explore_every=-1, tolerance=1e-12, corun_overhead_us=1e-9)
    profile_linear(ctl, 40.0, 5120.0, 4.0)
    B, Fl = 1.2e9, 240e-6 * 4e12 * 160
    d = ctl.decide(B, Fl, active_decode_seqs=64)
    assert d["cus_decode"] == 128 and abs(d["predicted_us"] - 300.0) < 1e-6
    d = ctl.decide(B, Fl, active_decode_seqs=64, decode_tail=True)
    assert d["mode"] == F.FLEX_MODE_CORUN and d["cus_decode"] == 96
    assert abs(d["predicted_us"] - 294.375) < 1e-6


def test_monotone_in_the_steps_work():
    ctl = F.Controller(granule=32, explore_every=-1, tolerance=1e-12)
    profile_linear(ctl, 36.0, 5600.0, 3.0)
    last = None
    for Fl in [2e10, 5e10, 1e11, 2e11, 4e11, 8e11]:   # more prefill work: decode share never grows
        d = ctl.decide(1.0e9, Fl, active_decode_seqs=64)
        if d["mode"] == F.FLEX_MODE_CORUN:
            assert last is None or d["cus_decode"] <= last
            last = d["cus_decode"]
    last = None
    for B in [2e8, 5e8, 1e9, 2e9, 4e9]:               # more decode work: decode share never shrinks
        d = ctl.decide(B, 1.5e11, active_decode_seqs=64)
        if d["mode"] == F.FLEX_MODE_CORUN:
            assert last is None or d["cus_decode"] >= last
            last = d["cus_decode"]


def test_saturated_decode_cedes_cus_and_backlog_takes_them():
    # decode saturates at 4800 GB/s from 160 CUs on: a wide band of equally fast
    # splits once prefill is small
    def fresh():
        c = F.Controller(granule=32, explore_every=-1, tolerance=0.05)
        profile_linear(c, 30.0, 4800.0, 3.0)
        return c
    B, Fl = 1.3e9, 2.0e10
    base = fresh().decide(B, Fl, active_decode_seqs=128)
    sat = fresh()
    sat.observe(160, B, 0.0, B / 4.9e12 * 1e3, 0.0)     # observed 4.9 TB/s >= 0.6 * 8 TB/s
    d_sat = sat.decide(B, Fl, active_decode_seqs=128)
    d_back = fresh().decide(B, Fl, pending_decode_seqs=1000, active_decode_seqs=128)
    assert d_sat["reason"] == F.FLEX_CTL_BW_SATURATED and d_back["reason"] == F.FLEX_CTL_BACKLOG
    assert d_sat["cus_decode"] <= base["cus_decode"] <= d_back["cus_decode"]
    assert d_sat["cus_decode"] < d_back["cus_decode"]
    # saturated decode never gets more CUs than saturation needs (within the band)
    assert d_sat["cus_decode"] <= 192
    # a prefill backlog (no bandwidth pressure observed) also takes the smallest
    # decode share of the band, the same choice as bandwidth pressure
    d_pre = fresh().decide(B, Fl, pending_prefill_tokens=100000, active_decode_seqs=128)
    assert d_pre["reason"] == F.FLEX_CTL_PREFILL_BACKLOG
    assert d_pre["cus_decode"] == d_sat["cus_decode"] <= base["cus_decode"]


def test_one_phase_runs_serial():
    ctl = F.Controller()
    for B, Fl, act in [(0.0, 1e11, 0), (1e9, 0.0, 5), (1e9, 1e11, 0)]:
        d = ctl.decide(B, Fl, active_decode_seqs=act)
        assert d["mode"] == F.FLEX_MODE_SERIAL and d["reason"] == F.FLEX_CTL_ONE_PHASE
        assert d["cus_decode"] == 256


def test_estimates_converge_to_observed_rates():
    ctl = F.Controller(alpha=0.25, explore_every=-1, granule=64)
    prior_d, prior_p = ctl.estimates()
    for _ in range(40):
        ctl.observe(128, 1.0e9, 1.0e11, 0.25, 0.2)       # 4000 GB/s, 500 TFLOP/s
    d, p = ctl.estimates()
    assert abs(d[1] - 4000.0) < 1e-9 and abs(p[1] - 500.0) < 1e-9   # first observation replaces the prior
    assert d[0] == prior_d[0] and p[2] == prior_p[2]                  # other splits untouched
    ctl.observe(128, 1.0e9, 1.0e11, 0.5, 0.4)            # one slower step moves the estimate by alpha
    d, p = ctl.estimates()
    assert abs(d[1] - (0.75 * 4000.0 + 0.25 * 2000.0)) < 1e-9


def test_exploration_visits_neighbours():
    # saturating decode: the best split is 128 (293 us; serial 341 us)
    ctl = F.Controller(granule=64, explore_every=4, tolerance=1e-12, corun_overhead_us=1e-9)
    profile_linear(ctl, 40.0, 5120.0, 4.0)
    picks = [ctl.decide(1e9, 1.5e11, active_decode_seqs=8) for _ in range(16)]
    for i, d in enumerate(picks, start=1):
        if i % 4 == 0:
            assert d["reason"] == F.FLEX_CTL_EXPLORE
        else:
            assert d["reason"] == F.FLEX_CTL_BEST
    best = picks[0]["cus_decode"]
    assert {picks[3]["cus_decode"], picks[7]["cus_decode"]} == {best - 64, best + 64}


def test_planted_mistake_is_caught():
    # An oracle that applies the bandwidth rule before the backlog rule must
    # disagree with the library somewhere on the parity sequence.
    class Swapped(OC.Controller):
        def decide(self, B, Fl, pending_prefill_tokens=0, pending_decode_seqs=0, active_decode_seqs=1):
            if self.last_bw >= self.o.sat_frac * self.o.hbm_gbps:
                pending_decode_seqs = 0
            return super().decide(B, Fl, pending_prefill_tokens, pending_decode_seqs, active_decode_seqs)
    lib = F.Controller(explore_every=-1)
    bad = Swapped(OC.CtlOpts(explore_every=-1))
    rng = random.Random(1)
    differ = False
    for _ in range(300):
        B, Fl = rng.uniform(5e8, 2e9), rng.uniform(2e10, 4e11)
        sig = dict(pending_decode_seqs=rng.randrange(0, 600), active_decode_seqs=100)
        a, b = lib.decide(B, Fl, **sig), bad.decide(B, Fl, **sig)
        differ |= (a["cus_decode"], a["reason"]) != (b["cus_decode"], b["reason"])
        cd = a["cus_decode"] if a["mode"] == F.FLEX_MODE_CORUN else 0
        obs = (cd, B, Fl, B / rng.uniform(3e12, 6e12) * 1e3, Fl / rng.uniform(2e14, 6e14) * 1e3)
        lib.observe(*obs)
        bad.observe(*obs)
    assert differ


def test_invalid_options_rejected():
    with pytest.raises(F.FlexAttnError):
        F.Controller(granule=96)          # does not divide 256
    with pytest.raises(F.FlexAttnError):
        F.Controller(alpha=1.5)
    ctl = F.Controller()
    with pytest.raises(F.FlexAttnError):
        ctl.observe(100, 1e9, 1e11, 0.1, 0.1)   # not a candidate split
    with pytest.raises(F.FlexAttnError):
        ctl.set_profile([64, 32], [1.0, 2.0], [1.0, 2.0])


def test_fused_form_follows_its_observed_ratio():
    # serial beats every split on this profile (no co-run gain): the one-launch
    # form is chosen while its ratio to the serial prediction is below 1
    ctl = F.Controller(granule=64, explore_every=4, tolerance=1e-12, corun_overhead_us=1000.0, fused_prior=0.8)
    profile_linear(ctl, 40.0, 5120.0, 4.0)
    B, Fl = 1.0e9, 1.5e11
    d1 = ctl.decide(B, Fl, active_decode_seqs=8, fused_available=True)
    serial_us = B / 5120e9 * 1e6 + Fl / 1024e12 * 1e6                 # 195.3 + 146.5 us
    assert d1["mode"] == F.FLEX_MODE_FUSED and d1["reason"] == F.FLEX_CTL_FUSED_FASTER
    assert abs(d1["predicted_us"] - 0.8 * serial_us) < 1e-9
    # without a one-launch form the same step runs serial
    d2 = ctl.decide(B, Fl, active_decode_seqs=8)
    assert d2["mode"] == F.FLEX_MODE_SERIAL and d2["reason"] == F.FLEX_CTL_SERIAL_FASTER
    # a fused step observed at 1.25 x the serial prediction: the first
    # observation replaces the prior, so serial wins from now on ...
    ctl.observe(256, B, Fl, 0.0, 0.0, fused=True, step_ms=1.25 * serial_us * 1e-3)
    # ... except on the explore turn that tries the form (decision 12: 12 // 4 = 3 mod 4)
    picks = [ctl.decide(B, Fl, active_decode_seqs=8, fused_available=True) for _ in range(14)]   # decisions 3..16
    turns = {i: d for i, d in enumerate(picks, start=3)}
    assert turns[12]["mode"] == F.FLEX_MODE_FUSED and turns[12]["reason"] == F.FLEX_CTL_EXPLORE
    assert abs(turns[12]["predicted_us"] - 1.25 * serial_us) < 1e-6
    for i, d in turns.items():
        if i != 12:
            assert d["mode"] == F.FLEX_MODE_SERIAL, (i, d)


def test_fused_must_beat_the_best_split():
    # co-run predicted 293 us, serial 341 us (saturating decode profile);
    # ratio 0.9 -> 307 us: the split stays; ratio 0.8 -> 273 us: fused
    def ctl(prior):
        c = F.Controller(granule=64, explore_every=-1, tolerance=1e-12, corun_overhead_us=1e-9, fused_prior=prior)
        profile_linear(c, 40.0, 5120.0, 4.0)
        return c
    B, Fl = 1.0e9, 1.5e11
    d = ctl(0.9).decide(B, Fl, active_decode_seqs=8, fused_available=True)
    assert d["mode"] == F.FLEX_MODE_CORUN and d["cus_decode"] == 128
    d = ctl(0.8).decide(B, Fl, active_decode_seqs=8, fused_available=True)
    assert d["mode"] == F.FLEX_MODE_FUSED and d["reason"] == F.FLEX_CTL_FUSED_FASTER


def test_fused_ratio_is_relative_to_observed_serial_steps():
    # launch gaps outside the phase times: a serial step observed at 1.5 x its
    # prediction and a fused step at 1.2 x make the fused form 0.8 x serial
    ctl = F.Controller(granule=64, explore_every=-1, tolerance=1e-12, corun_overhead_us=1000.0, fused_prior=2.0)
    profile_linear(ctl, 40.0, 5120.0, 4.0)
    B, Fl = 1.0e9, 1.5e11
    serial_us = B / 5120e9 * 1e6 + Fl / 1024e12 * 1e6
    assert ctl.decide(B, Fl, active_decode_seqs=8, fused_available=True)["mode"] == F.FLEX_MODE_SERIAL
    ctl.observe(0, B, Fl, 0.0, 0.0, step_ms=1.5 * serial_us * 1e-3)            # step time only
    ctl.observe(0, B, Fl, 0.0, 0.0, fused=True, step_ms=1.2 * serial_us * 1e-3)
    d = ctl.decide(B, Fl, active_decode_seqs=8, fused_available=True)
    assert d["mode"] == F.FLEX_MODE_FUSED and d["reason"] == F.FLEX_CTL_FUSED_FASTER
    assert abs(d["predicted_us"] - 0.8 * serial_us) < 1e-9
    # step-time-only observations leave the phase-rate estimates alone
    assert abs(ctl.decide(B, Fl, active_decode_seqs=8)["predicted_us"] - serial_us) < 1e-9


# ---------------------------------------------------------------------------
# Time-slice scheduler (flex_ts_*)

def test_timeslice_worked_example():
    """share 1/4 (decode when 3 * t_dec <= t_pre), decode steps 1 ms, prefill
    steps 2 ms, whole history; worked by hand, (t_dec, t_pre) after each step:
    D (1,0), P (1,2), P (1,4), D (2,4), P (2,6), D (3,6), P (3,8), P (3,10)."""
    ts = F.TimeSlice(decode_share=0.25)
    seq = []
    for _ in range(8):
        ph = ts.next(True, True)
        seq.append("D" if ph == F.FLEX_TS_DECODE else "P")
        ts.observe(ph, 1.0 if ph == F.FLEX_TS_DECODE else 2.0)
    assert "".join(seq) == "DPPDPDPP"
    assert ts.totals() == (3.0, 10.0)
    ts.close()


@pytest.mark.parametrize("share", [0.2, 0.5, 0.8])
@pytest.mark.parametrize("dur", [(0.1, 0.25), (0.3, 0.07), (1.0, 1.0)])
def test_timeslice_share_converges(share, dur):
    """Both phases always ready, whole history: after every step decode's share of
    the total time is within one step's duration (relative to the total) of the target."""
    ts = F.TimeSlice(decode_share=share)
    td = tp = 0.0
    for i in range(400):
        ph = ts.next(True, True)
        ts.observe(ph, dur[ph])
        if ph == F.FLEX_TS_DECODE:
            td += dur[0]
        else:
            tp += dur[1]
        if i > 10:
            assert abs(td / (td + tp) - share) <= max(dur) / (td + tp) + 1e-12
    ts.close()


def test_timeslice_one_ready_phase_and_errors():
    ts = F.TimeSlice(decode_share=0.9)
    for _ in range(5):
        assert ts.next(False, True) == F.FLEX_TS_PREFILL
        ts.observe(F.FLEX_TS_PREFILL, 1.0)
    assert ts.next(True, False) == F.FLEX_TS_DECODE
    with pytest.raises(F.FlexAttnError):
        ts.next(False, False)
    with pytest.raises(F.FlexAttnError):
        ts.observe(7, 1.0)
    with pytest.raises(F.FlexAttnError):
        ts.observe(F.FLEX_TS_DECODE, -1.0)
    with pytest.raises(F.FlexAttnError):
        F.TimeSlice(decode_share=1.0)
    with pytest.raises(F.FlexAttnError):
        F.TimeSlice(decode_share=0.5, decay=1.5)
    ts.close()


@pytest.mark.parametrize("seed", range(4))
def test_timeslice_matches_rederivation(seed):
    """Random readiness and durations, a decaying window: every choice and the
    final totals equal the re-derivation's, exactly."""
    rng = random.Random(seed)
    share, decay = rng.uniform(0.05, 0.95), rng.choice([1.0, 0.9, 0.5])
    a, b = F.TimeSlice(share, decay), OC.TimeSlice(share, decay)
    for _ in range(500):
        dr, pr = bool(rng.random() < 0.9), bool(rng.random() < 0.7)
        if not (dr or pr):
            continue
        pa, pb = a.next(dr, pr), b.next(dr, pr)
        assert pa == pb
        ms = rng.expovariate(1.0 / (0.2 if pa == OC.TS_DECODE else 0.5))
        a.observe(pa, ms)
        b.observe(pb, ms)
    assert a.totals() == (b.t_dec, b.t_pre)
    a.close()


def test_timeslice_decay_forgets():
    """decay 0.5: after a long prefill-only stretch the decode total has decayed
    to nothing, so decode runs first when both become ready again."""
    ts = F.TimeSlice(decode_share=0.1, decay=0.5)
    for _ in range(3):
        ts.observe(F.FLEX_TS_DECODE, 10.0)
    for _ in range(60):
        ts.observe(F.FLEX_TS_PREFILL, 0.01)
    d, p = ts.totals()
    assert d < 1e-15 and p > 0
    assert ts.next(True, True) == F.FLEX_TS_DECODE
    ts.close()


def test_controller_seeds_from_the_committed_cu_sweep():
    """The measured CU sweep of the mixed step (profiles/cusweep_mixed.json)
    is the controller's alone-phase profile (flex_ctl_set_profile)."""
    from paper_2606_04415_amd.serve_sim import measure_profile
    cus, dec, pre = measure_profile()
    assert cus == [64, 128, 192, 256] and all(x > 0 for x in dec + pre)
    ctl = F.Controller()
    ctl.set_profile(cus, dec, pre)
    d_est, p_est = ctl.estimates()
    assert all(x > 0 for x in d_est + p_est)
    d = ctl.decide(1.2e9, 1.5e11, active_decode_seqs=128)
    assert d["mode"] in (F.FLEX_MODE_SERIAL, F.FLEX_MODE_CORUN) and d["predicted_us"] > 0


def test_latent_sweep_seeds_a_serial_decision():
    """Seeded with the measured CU sweep of the latent step
    (profiles/cusweep_mla.json), the controller runs that step's work
    serially: its decode loses most of its speed on a small CU share, so no
    split beats prefill then decode on the whole device (the sweep's own
    co-run steps agree)."""
    import json
    import os
    from paper_2606_04415_amd.cusweep import PROFILE_DIR, profile_from
    path = os.path.join(PROFILE_DIR, "cusweep_mla.json")
    with open(path) as f:
        sweep = json.load(f)
    assert sweep["serial_us"] < sweep["best_split"]["us"]
    cus, dec, pre = profile_from(path)
    assert cus == [32, 64, 96, 128, 160, 192, 224, 256]
    ctl = F.Controller()
    ctl.set_profile(cus, dec, pre)
    d = ctl.decide(sweep["decode_bytes"], sweep["prefill_flops"], active_decode_seqs=256)
    assert d["mode"] == F.FLEX_MODE_SERIAL
    # the mixed step's sweep, same rule: a co-run split
    cus_m, dec_m, pre_m = profile_from(os.path.join(PROFILE_DIR, "cusweep_mixed.json"))
    ctl_m = F.Controller()
    ctl_m.set_profile(cus_m, dec_m, pre_m)
    with open(os.path.join(PROFILE_DIR, "cusweep_mixed.json")) as f:
        mixed = json.load(f)
    dm = ctl_m.decide(mixed["decode_bytes"], mixed["prefill_flops"], active_decode_seqs=128)
    assert dm["mode"] == F.FLEX_MODE_CORUN
