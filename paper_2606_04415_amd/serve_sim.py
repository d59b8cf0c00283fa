"""Step-level serving simulation: serial vs a fixed co-run split vs the online controller.

The paper evaluates dynamic prefill/decode co-location against static
co-location and disaggregation by end-to-end serving latency (TTFT, TPOT) on
1K-input/1K-output and 1K-input/4K-output request mixes (Sec. 4.1; Tables 3
and 4). This tool replays one synthetic request stream per mix through the
library on one GPU, step by step, under four policies, and reports the
step-time distribution and TTFT / TPOT proxies:

* serial      every step runs prefill then decode on all CUs;
* fixed       a step with both phases co-runs on a fixed CU split (static
              co-location), otherwise serial;
* controller  flex_ctl_* picks each step's mode (serial, a co-run split, or
              the one-launch form) from the step's work and queue signals,
              observing every step's phase times (dynamic co-location;
              Sec. 3.3, Sec. 3.4);
* fused       a step with both phases runs as one launch whose work-groups
              interleave the phases (no CU masks), otherwise serial;
* timeslice   temporal multiplexing instead of co-location inside a step:
              each step runs one phase alone on all CUs (all decodes, or
              prompt chunks), flex_ts_* choosing the phase so that decode's
              share of the recent device time tracks a target
              (`timeslice:0.3` = 30%; Sec. 3 and Sec. 3.4, and the time-slice
              ratio of Sec. 4).

The stream is defined in steps, not in time: requests arrive at given steps,
are admitted while there is room, and are prefilled in chunks of at most
`chunk` tokens per step (oldest first) before they decode one token per step.
So every co-location policy runs exactly the same sequence of batches; only
the time each step takes differs (timeslice splits each such batch's phases
over separate steps). A step is the KV append of its new tokens plus the
attention of the mixed batch (GPU time, HIP events on the issuing stream,
with no per-phase events inside: the controller's phase times come from an
untimed repeat of the step's attention); plan building and upload are host
work outside it, timed per step (plan_host_ms) and added in series to the
device time in total_with_plan_ms (the run if planning did not overlap the
previous step's GPU work, which a serving engine would do). Request time stamps use
the running sum of step times: TTFT = end of the step that finishes a
request's prompt minus the time it arrived; TPOT = the time from a request's
previous token (or the end of its prompt) to each of its decode tokens, over
all decode tokens of the run (under the co-location policies every decoding
request gets one token per step, so this is that step's time). Synthetic: random K/V contents, Qwen2.5-7B attention
geometry (28/4 heads x 128, page 16), lengths drawn from a seeded generator.

    python -m paper_2606_04415_amd.serve_sim --mix 1k1k --steps 300
"""
from __future__ import annotations

import argparse
import json
import math
import os
import random
import sys
import time
from dataclasses import dataclass, field
from typing import Dict, List, Optional

MIXES = {
    # prompt and output length ranges (uniform, inclusive)
    "1k1k": ((768, 1280), (768, 1280)),
    "1k4k": ((768, 1280), (3072, 5120)),
    # long contexts: steps the size of the mixed benchmark step (2048-token
    # chunks on ~4K prompts beside ~128 decodes over 2K-11K keys)
    "long": ((3072, 5120), (2048, 6144)),
}
# per-mix batch limits (max active, warm, burst) where they differ from the flags' defaults
MIX_LIMITS = {"long": (128, 112, 24)}
HQ, HKV, D, P = 28, 4, 128, 16


@dataclass
class Req:
    rid: int
    prompt: int
    out: int
    arrival_step: int
    arrival_ms: float = 0.0
    prefilled: int = 0
    generated: int = 0
    pages: List[int] = field(default_factory=list)
    last_tok_ms: float = 0.0
    first_ms: Optional[float] = None
    finish_ms: Optional[float] = None

    @property
    def ctx(self) -> int:
        """Keys in the cache (prompt tokens processed + generated tokens after the first)."""
        return self.prefilled + max(0, self.generated - 1)


def make_stream(mix: str, steps: int, seed: int, warm: int, burst: int, burst_every: int,
                rate: float) -> List[Req]:
    """Warm requests (already decoding at step 0, at random progress), bursts of
    new prompts every burst_every steps, and Poisson arrivals at `rate` per step."""
    (p_lo, p_hi), (o_lo, o_hi) = MIXES[mix]
    rng = random.Random(seed)
    reqs: List[Req] = []
    for _ in range(warm):
        r = Req(len(reqs), rng.randint(p_lo, p_hi), rng.randint(o_lo, o_hi), arrival_step=-1)
        r.prefilled = r.prompt
        r.generated = rng.randint(1, r.out - 1)
        reqs.append(r)
    for s in range(steps):
        n = burst if burst_every and s % burst_every == 0 else 0
        # Poisson arrivals by inversion
        u, k, pk = rng.random(), 0, math.exp(-rate)
        cum = pk
        while u > cum and k < 100:
            k += 1
            pk *= rate / k
            cum += pk
        for _ in range(n + k):
            reqs.append(Req(len(reqs), rng.randint(p_lo, p_hi), rng.randint(o_lo, o_hi), arrival_step=s))
    return reqs


def simulate(mix: str, policy: str, args, profile=None) -> Dict:
    import torch
    from . import flexattn as F

    dev = torch.device("cuda:0")
    if mix in MIX_LIMITS and args.per_mix_limits:
        args = argparse.Namespace(**vars(args))
        args.max_active, args.warm, args.burst = MIX_LIMITS[mix]
    reqs = make_stream(mix, args.steps, args.seed, args.warm, args.burst, args.burst_every, args.rate)
    max_ctx = MIXES[mix][0][1] + MIXES[mix][1][1] + 1
    pages_per_req = -(-max_ctx // P)
    n_pages = args.max_active * pages_per_req + 1
    gen = torch.Generator(device=dev).manual_seed(args.seed)
    k_cache = torch.randn((n_pages, P, HKV, D), generator=gen, device=dev).to(torch.bfloat16)
    v_cache = torch.randn((n_pages, P, HKV, D), generator=gen, device=dev).to(torch.bfloat16)
    free_pages = list(range(n_pages - 1, 0, -1))          # page 0 is a spare for unused entries
    shape = F.make_shape(HQ, HKV, D, D, P, 1.0 / math.sqrt(D), False)
    caller = torch.cuda.Stream()
    # One co-run pair open at a time, recreated when the split changes: every
    # open pair holds two streams, and HIP serves a process's streams from a
    # few hardware queues (4 here), so with several pairs open the phase
    # streams of one pair can share a queue and run one after the other
    # (measured: co-run steps 1.6x longer with seven pairs open). The switch
    # is host work, timed with the planning.
    pair = {"cd": None, "obj": None}

    def corun_for(cd):
        if pair["cd"] != cd:
            if pair["obj"] is not None:
                pair["obj"].close()
            pair["obj"], pair["cd"] = F.Corun(256 - cd, cd), cd
        return pair["obj"]
    corun_for(args.fixed_decode_cus if policy == "fixed" else 128)   # set-up, untimed
    ctl = None
    ts = None
    if policy.startswith("timeslice"):
        share = float(policy.split(":")[1]) if ":" in policy else args.decode_share
        ts = F.TimeSlice(share, getattr(args, "ts_decay", 0.9))
    phase_ms: Dict[str, float] = {}   # device time of decode-only, prefill-only and mixed steps
    prefill_tokens = 0
    if policy == "controller":
        ctl = F.Controller()
        if profile:
            ctl.set_profile(*profile)
    q_pool = torch.randn((args.chunk + args.max_active + 8, HQ, D), generator=gen, device=dev).to(torch.bfloat16)
    out_pool = torch.empty((args.chunk + args.max_active + 8, HQ, D), dtype=torch.bfloat16, device=dev)
    kn_pool = torch.randn((args.chunk + args.max_active + 8, HKV, D), generator=gen, device=dev).to(torch.bfloat16)
    vn_pool = torch.randn((args.chunk + args.max_active + 8, HKV, D), generator=gen, device=dev).to(torch.bfloat16)

    waiting: List[Req] = []
    active: List[Req] = []
    nxt = 0
    clock = 0.0
    step_ms: List[float] = []
    plan_ms: List[float] = []
    tok_ms: List[float] = []   # time since the previous token, for every decode token
    splits: Dict[str, int] = {}
    reasons: Dict[int, int] = {}
    done: List[Req] = []
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e_mid = torch.cuda.Event(enable_timing=True)   # after the append: the attention alone follows

    for step in range(args.steps):
        while nxt < len(reqs) and reqs[nxt].arrival_step <= step:
            r = reqs[nxt]
            r.arrival_ms = clock
            waiting.append(r)
            nxt += 1
        while waiting and len(active) < args.max_active and len(free_pages) >= pages_per_req:
            active.append(waiting.pop(0))
        # batch: decodes, then prompt chunks oldest first
        ns, ls, members = [], [], []
        budget = args.chunk
        for r in active:
            if r.prefilled == r.prompt:
                ns.append(1)
                ls.append(r.prefilled + r.generated)       # the new token's key is in the cache
                members.append((r, 1))
        for r in active:
            if r.prefilled < r.prompt and budget > 0:
                c = min(budget, r.prompt - r.prefilled)
                budget -= c
                ns.append(c)
                ls.append(r.prefilled + c)
                members.append((r, c))
        if ts is not None and members:
            has_dec = any(n == 1 and r.prefilled == r.prompt for r, n in members)
            has_pre = len(members) > sum(1 for r, n in members if n == 1 and r.prefilled == r.prompt)
            phase = ts.next(has_dec, has_pre)
            keep = [i for i, (r, n) in enumerate(members)
                    if (n == 1 and r.prefilled == r.prompt) == (phase == F.FLEX_TS_DECODE)]
            if phase == F.FLEX_TS_DECODE:
                budget = args.chunk                      # no prompt tokens run this step
            ns, ls, members = [ns[i] for i in keep], [ls[i] for i in keep], [members[i] for i in keep]
        if not members:
            step_ms.append(0.0)
            continue
        for (r, n), L in zip(members, ls):
            need = -(-L // P)
            while len(r.pages) < need:
                r.pages.append(free_pages.pop())
        B = len(members)
        max_pages = max(len(r.pages) for r, _ in members)
        bt = torch.zeros((B, max_pages), dtype=torch.int32)
        for i, (r, _) in enumerate(members):
            bt[i, :len(r.pages)] = torch.tensor(r.pages, dtype=torch.int32)
        qsl = [0]
        for n in ns:
            qsl.append(qsl[-1] + n)
        T = qsl[-1]
        slots = []
        for (r, n), L in zip(members, ls):
            for pos in range(L - n, L):
                slots.append(r.pages[pos // P] * P + pos % P)
        n_dec = sum(1 for n in ns if n == 1)
        pend_prefill = sum(r.prompt - r.prefilled for r in waiting + active) - (args.chunk - budget)
        # the policy's choice (host planning and upload are timed: plan_host_ms)
        t_plan = time.perf_counter()
        probe = F.PagedAttention(shape, F.make_opts(), qsl, ls, max_pages)
        info = probe.plan.info
        mode, cd = F.FLEX_MODE_SERIAL, 0
        both = info["n_decode_items"] > 0 and info["n_prefill_items"] > 0
        if policy == "fixed" and both:
            mode, cd = F.FLEX_MODE_CORUN, args.fixed_decode_cus
        elif policy == "fused" and both:
            mode = F.FLEX_MODE_FUSED
        elif policy == "controller":
            d = ctl.decide(info["decode_bytes"], info["prefill_flops"], pending_prefill_tokens=max(0, pend_prefill),
                           pending_decode_seqs=len(waiting), active_decode_seqs=n_dec,
                           fused_available=getattr(args, "controller_fused", True) and info["n_fused_wgs"] > 0,
                           decode_tail=True)   # grouped-query co-run plans form a decode tail
            reasons[d["reason"]] = reasons.get(d["reason"], 0) + 1
            if d["mode"] == F.FLEX_MODE_CORUN:
                mode, cd = F.FLEX_MODE_CORUN, d["cus_decode"]
            elif d["mode"] == F.FLEX_MODE_FUSED:
                mode = F.FLEX_MODE_FUSED
        if mode == F.FLEX_MODE_SERIAL:
            pa = probe
        elif mode == F.FLEX_MODE_FUSED:
            pa = F.PagedAttention(shape, F.make_opts(wg_per_cu=2), qsl, ls, max_pages)
        else:
            pa = F.PagedAttention(shape, F.make_opts(cus_decode=cd), qsl, ls, max_pages)
        # (SERIAL uses a pair only for its phase timing: whichever is open)
        corun = corun_for(cd if mode == F.FLEX_MODE_CORUN else (pair["cd"] or 128))
        plan_ms.append((time.perf_counter() - t_plan) * 1e3)
        key = {F.FLEX_MODE_SERIAL: "serial", F.FLEX_MODE_FUSED: "fused"}.get(mode, f"{256 - cd}:{cd}")
        if ts is not None:
            key = "decode" if phase == F.FLEX_TS_DECODE else "prefill"
        splits[key] = splits.get(key, 0) + 1
        d_bt = bt.to(dev)
        d_sl = torch.tensor(ls, dtype=torch.int32, device=dev)
        d_qsl = torch.tensor(qsl, dtype=torch.int32, device=dev)
        d_slots = torch.tensor(slots, dtype=torch.int32, device=dev)
        q, out = q_pool[:T], out_pool[:T]
        args_ = pa.args(q, k_cache, v_cache, d_bt, d_sl, d_qsl, out)
        app = F.make_append_args(kn_pool[:T], vn_pool[:T], d_slots, k_cache, v_cache)
        torch.cuda.synchronize()
        # the step, timed with no phase events (recording them adds ~10 us)
        e0.record(caller)
        F.flex_attn_kv_append(shape, app, stream=caller.cuda_stream)
        e_mid.record(caller)
        F.flex_attn_mixed(pa.plan, args_, mode, stream=caller.cuda_stream, corun=corun)
        e1.record(caller)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        attn_ms = e_mid.elapsed_time(e1)
        if ctl is not None and mode == F.FLEX_MODE_FUSED:
            ctl.observe(0, info["decode_bytes"], info["prefill_flops"], 0.0, 0.0, fused=True, step_ms=attn_ms)
        elif ctl is not None:
            # the controller's phase times: the same attention once more, untimed,
            # with phase events (it recomputes the same outputs)
            corun.set_timing(True)
            F.flex_attn_mixed(pa.plan, args_, mode, stream=caller.cuda_stream, corun=corun)
            pre_ms, dec_ms = corun.timing_read()
            corun.set_timing(False)
            # (a co-run step's timed decode phase leaves out the plan's decode tail)
            pinfo = pa.plan.info
            timed_bytes = pinfo["decode_bytes"] - (pinfo["decode_tail_bytes"] if mode == F.FLEX_MODE_CORUN else 0.0)
            ctl.observe(cd if mode == F.FLEX_MODE_CORUN else 0, timed_bytes, info["prefill_flops"],
                        dec_ms[-1] if dec_ms else 0.0, pre_ms[-1] if pre_ms else 0.0,
                        step_ms=attn_ms if mode == F.FLEX_MODE_SERIAL else 0.0)
        if ts is not None:
            ts.observe(phase, ms)
        n_dec_tok = sum(1 for r, n in members if n == 1 and r.prefilled == r.prompt)
        kind = "decode" if n_dec_tok == len(members) else "prefill" if n_dec_tok == 0 else "mixed"
        phase_ms[kind] = phase_ms.get(kind, 0.0) + ms
        clock += ms
        step_ms.append(ms)
        # advance the requests
        for r, n in members:
            if n == 1 and r.prefilled == r.prompt:
                r.generated += 1
                tok_ms.append(clock - r.last_tok_ms)
                r.last_tok_ms = clock
            else:
                r.prefilled += n
                prefill_tokens += n
                if r.prefilled == r.prompt:
                    r.generated = 1
                    r.first_ms = clock
                    r.last_tok_ms = clock
            if r.generated >= r.out:
                r.finish_ms = clock
                free_pages.extend(r.pages)
                r.pages = []
                done.append(r)
        active = [r for r in active if r.finish_ms is None]
    if pair["obj"] is not None:
        pair["obj"].close()
    if ts is not None:
        ts.close()

    def pct(xs, p):
        xs = sorted(xs)
        return xs[min(len(xs) - 1, int(p * len(xs)))] if xs else None

    busy = [x for x in step_ms if x > 0]
    plan_total = sum(plan_ms)
    ttft = [r.first_ms - r.arrival_ms for r in reqs[:nxt] if r.first_ms is not None and r.arrival_step >= 0]
    res = {"mix": mix, "policy": policy, "steps": args.steps, "total_ms": round(clock, 3),
           "step_ms": {"mean": round(sum(busy) / max(1, len(busy)), 4), "p50": pct(busy, 0.5), "p90": pct(busy, 0.9),
                       "max": max(busy) if busy else None},
           "ttft_ms": {"n": len(ttft), "p50": pct(ttft, 0.5), "p90": pct(ttft, 0.9),
                       "mean": round(sum(ttft) / len(ttft), 3) if ttft else None},
           "tpot_ms": {"tokens": len(tok_ms), "mean": round(sum(tok_ms) / len(tok_ms), 4) if tok_ms else None,
                       "p90": pct(tok_ms, 0.9)},
           "throughput": {"decode_tok_per_s": round(len(tok_ms) / clock * 1e3, 1) if clock else None,
                          "prefill_tok_per_s": round(prefill_tokens / clock * 1e3, 1) if clock else None},
           "device_ms": {k: round(v, 3) for k, v in phase_ms.items()},
           # host planning (plan build + upload, incl. the policy's probe plan) per step: a serving
           # engine overlaps it with the previous step's GPU work; total_with_plan_ms is the run if it
           # did not (host and device time in series)
           "plan_host_ms": {"mean": round(plan_total / max(1, len(plan_ms)), 4), "p90": pct(plan_ms, 0.9)},
           "total_with_plan_ms": round(clock + plan_total, 3),
           "splits": splits}
    if ctl is not None:
        res["reasons"] = {str(k): v for k, v in sorted(reasons.items())}
    return res


def measure_profile(reps: int = 10, remeasure: bool = False):
    """Alone phase rates on 64..256 CUs (quarters, the controller's default
    candidate splits) for the mixed step, to seed the controller: the
    committed CU sweep (profiles/cusweep_mixed.json) when present, else
    measured now."""
    from .cusweep import PROFILE_DIR, profile_from, sweep
    path = os.path.join(PROFILE_DIR, "cusweep_mixed.json")
    if os.path.exists(path) and not remeasure:
        cus, dec, pre = profile_from(path)
        keep = [i for i, c in enumerate(cus) if c % 64 == 0]
        return [cus[i] for i in keep], [dec[i] for i in keep], [pre[i] for i in keep]
    r = sweep("mixed", reps=reps, pools=2, counts=[64, 128, 192, 256], corun=False)
    return profile_from(r)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--mix", default="all", choices=["1k1k", "1k4k", "long", "all"])
    ap.add_argument("--no-per-mix-limits", dest="per_mix_limits", action="store_false",
                    help="use the flags' batch limits for every mix")
    ap.add_argument("--policies", default="serial,fixed,controller,fused")
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--warm", type=int, default=224, help="requests already decoding at step 0")
    ap.add_argument("--max-active", type=int, default=256)
    ap.add_argument("--chunk", type=int, default=2048, help="prefill tokens per step")
    ap.add_argument("--burst", type=int, default=64, help="prompts arriving together every --burst-every steps")
    ap.add_argument("--burst-every", type=int, default=100)
    ap.add_argument("--rate", type=float, default=0.2, help="Poisson arrivals per step")
    ap.add_argument("--fixed-decode-cus", type=int, default=96)
    ap.add_argument("--no-profile", action="store_true", help="controller starts from its prior only")
    ap.add_argument("--remeasure-profile", action="store_true",
                    help="measure the phase profile now instead of reading profiles/cusweep_mixed.json")
    ap.add_argument("--decode-share", type=float, default=0.5,
                    help="timeslice policy: target decode share of device time (or name it: timeslice:0.3)")
    ap.add_argument("--ts-decay", type=float, default=0.9,
                    help="timeslice policy: weight kept by past device time per step (window ~ 1 / (1 - decay))")
    ap.add_argument("--no-controller-fused", dest="controller_fused", action="store_false",
                    help="the controller chooses between serial and co-run only")
    args = ap.parse_args()
    profile = None if args.no_profile else measure_profile(remeasure=args.remeasure_profile)
    if profile:
        print(json.dumps({"profile": {"cus": profile[0], "decode_GBps": profile[1], "prefill_TFLOPs": profile[2]}}),
              flush=True)
    mixes = list(MIXES) if args.mix == "all" else [args.mix]
    for mix in mixes:
        for pol in args.policies.split(","):
            t0 = time.perf_counter()
            r = simulate(mix, pol, args, profile)
            r["host_s"] = round(time.perf_counter() - t0, 1)
            print(json.dumps(r), flush=True)
            print(f"{mix} {pol}: total {r['total_ms']:.1f} ms", file=sys.stderr, flush=True)


if __name__ == "__main__":
    main()
