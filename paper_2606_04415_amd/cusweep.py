"""CU sweep and co-run split optimiser for one mixed batch on one MI355X.

The paper's starting observation (Sec. 2, Fig. 2) is that decode attention
stops gaining bandwidth well before it has every compute unit, while prefill
keeps scaling with compute units; phase-aware co-location gives each phase
the share it can use. This tool measures both curves on this device with the
library's own CU-masked streams, then the co-run step time of every split,
and reports the best split next to serial execution:

    python -m paper_2606_04415_amd.cusweep --workload mixed

Decode is timed alone on a stream masked to c CUs with a plan partitioned for
c CUs (all its ranges, a decode tail included); prefill alone on c CUs with
the plan for a c-CU prefill share; a co-run step on (256 - c_d, c_d), with
the plan's decode tail where it forms one. Counts step
in eighths of the device (the co-run mask granularity). Prints one JSON
object on stdout.
"""
from __future__ import annotations

import argparse
import json
import os
import sys


def _time_on(stream_handle, fn, reps, warmup=30, settle_ms=100.0, budget_ms=1500.0):
    """Mean us per call of fn over reps calls on the stream, after warmup calls
    and settle_ms of further untimed calls (the device raises its clock over
    the first MFMA-heavy launches after idle). Slow calls get fewer warmup
    calls and repetitions, so that one measurement stays near budget_ms."""
    import time
    import torch
    s = torch.cuda.ExternalStream(stream_handle) if stream_handle else torch.cuda.current_stream()
    t0 = time.perf_counter()
    fn()
    torch.cuda.synchronize()
    once_ms = (time.perf_counter() - t0) * 1e3
    fit = max(3, int(budget_ms / max(once_ms, 1e-3) / 2))
    warmup, reps = min(warmup, fit), min(reps, fit)
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < settle_ms * 1e-3:
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s)
    for i in range(reps):
        fn(i)
    e1.record(s)
    e1.synchronize()
    return e0.elapsed_time(e1) / reps * 1e3   # us


def sweep(workload: str = "mixed", reps: int = 20, pools: int = 4, seed: int = 0, counts=None, corun: bool = True,
          check_outputs: bool = False):
    """Phase curves and co-run step times (see the module text). With
    check_outputs, each split's plan also runs once serially and once
    co-run into separate outputs, and `corun_bitwise_equals_serial` records
    whether the two are bit-identical."""
    import torch
    from . import flexattn as F
    from .workloads import WORKLOADS, algorithmic_work, make_batch

    w = WORKLOADS[workload]
    b = make_batch(w, seed=seed, poison=False)
    work = algorithmic_work(w, b.extra["ns"], b.extra["ls"])
    dev = torch.device("cuda:0")
    q = b.q.to(dev)
    kv = [(b.k_cache.to(dev), b.v_cache.to(dev) if b.v_cache is not None else None) for _ in range(max(1, pools))]
    bt, sl, qsl = b.block_table.to(dev), b.seq_lens.to(dev), b.query_start_loc.to(dev)
    shape = F.make_shape(w.num_q_heads, w.num_kv_heads, w.head_dim_qk, w.head_dim_v, w.page_size,
                         w.sm_scale, w.v_aliases_k)
    total = torch.cuda.get_device_properties(0).multi_processor_count
    step = total // 8
    counts = sorted(counts) if counts else list(range(step, total + 1, step))

    def plan_for(cus_decode):
        pa = F.PagedAttention(shape, F.make_opts(cus_decode=cus_decode), b.query_start_loc.tolist(),
                              b.seq_lens.tolist(), b.block_table.shape[1])
        out, _ = pa.alloc_out(q)
        return pa, [pa.args(q, k, v, bt, sl, qsl, out) for k, v in kv]

    dec_bytes, pre_flops = work["decode"]["bytes"], work["prefill"]["flops"]
    res = {"workload": workload, "cus_total": total, "decode_bytes": dec_bytes, "prefill_flops": pre_flops,
           "decode": {}, "prefill": {}, "corun_step_us": {}}
    for c in counts:
        pa, args = plan_for(c if c < total else 0)                 # decode share of c CUs
        pa_p, args_p = plan_for(total - c if c < total else 0)     # prefill share of c CUs
        corun_d = F.Corun(total - c, c) if c < total else None
        corun_p = F.Corun(c, total - c) if c < total else None
        sd = corun_d.streams()[1] if corun_d else None
        sp = corun_p.streams()[0] if corun_p else None
        if dec_bytes:
            us = _time_on(sd, lambda i=0: F.flex_attn_decode(pa.plan, args[i % len(args)], stream=sd), reps)
            res["decode"][c] = {"us": round(us, 2), "GBps": round(dec_bytes / (us * 1e-6) / 1e9, 1)}
        if pre_flops:
            us = _time_on(sp, lambda i=0: F.flex_attn_prefill(pa_p.plan, args_p[i % len(args_p)], stream=sp), reps)
            res["prefill"][c] = {"us": round(us, 2), "TFLOPs": round(pre_flops / (us * 1e-6) / 1e12, 1)}
        for cr in (corun_d, corun_p):
            if cr:
                cr.close()
        print(f"cus {c}: decode {res['decode'].get(c)} prefill {res['prefill'].get(c)}", file=sys.stderr, flush=True)
    if dec_bytes and pre_flops and corun:
        # steps issued from a stream of their own (the legacy default stream
        # would synchronize with the co-run streams at every step)
        caller = torch.cuda.Stream()
        cs = caller.cuda_stream
        if check_outputs:
            res["corun_bitwise_equals_serial"] = {}
        res["corun_phases_us"] = {}
        res["decode_tail_frac"] = {}
        for cd in [c for c in counts if c < total]:
            print(f"co-run prefill {total - cd} / decode {cd}: measuring", file=sys.stderr, flush=True)
            pa, args = plan_for(cd)
            inf = pa.plan.info
            res["decode_tail_frac"][cd] = round(inf["decode_tail_bytes"] / inf["decode_bytes"], 4) if inf["decode_bytes"] else 0.0
            cr = F.Corun(total - cd, cd)
            if check_outputs:
                outs = []
                for mode in (F.FLEX_MODE_SERIAL, F.FLEX_MODE_CORUN):
                    o, _ = pa.alloc_out(q)
                    a = pa.args(q, kv[0][0], kv[0][1], bt, sl, qsl, o)
                    F.flex_attn_mixed(pa.plan, a, mode, stream=cs, corun=cr)
                    torch.cuda.synchronize()
                    outs.append(o)
                res["corun_bitwise_equals_serial"][cd] = bool(torch.equal(outs[0].view(torch.int16),
                                                                          outs[1].view(torch.int16)))
            us = _time_on(cs, lambda i=0: F.flex_attn_mixed(pa.plan, args[i % len(args)], F.FLEX_MODE_CORUN,
                                                             stream=cs, corun=cr), reps)
            # each phase's own duration in the co-run step (events on its stream)
            cr.set_timing(True)
            for i in range(min(reps, 5)):
                F.flex_attn_mixed(pa.plan, args[i % len(args)], F.FLEX_MODE_CORUN, stream=cs, corun=cr)
            torch.cuda.synchronize()
            pre, dec = cr.timing_read()
            cr.set_timing(False)
            cr.close()
            res["corun_step_us"][cd] = round(us, 2)
            res["corun_phases_us"][cd] = {"prefill": round(sum(pre) / len(pre) * 1e3, 2),
                                          "decode": round(sum(dec) / len(dec) * 1e3, 2)}
            print(f"co-run prefill {total - cd} / decode {cd}: {us:.1f} us (phases {res['corun_phases_us'][cd]})",
                  file=sys.stderr, flush=True)
        pa, args = plan_for(0)
        res["serial_us"] = round(_time_on(cs, lambda i=0: F.flex_attn_mixed(pa.plan, args[i % len(args)],
                                                                            F.FLEX_MODE_SERIAL, stream=cs), reps), 2)
        best = min(res["corun_step_us"], key=res["corun_step_us"].get)
        res["best_split"] = {"cus_prefill": total - best, "cus_decode": best, "us": res["corun_step_us"][best],
                             "speedup_vs_serial": round(res["serial_us"] / res["corun_step_us"][best], 4)}
        # what the phase curves alone predict per split: the slower phase, or, when
        # the split's plan has a decode tail, the prefill plus decode's rest at the
        # rate decode reaches on all CUs
        pred = {}
        for cd in res["corun_step_us"]:
            if total - cd not in res["prefill"]:
                continue
            t_dec, t_pre = res["decode"][cd]["us"], res["prefill"][total - cd]["us"]
            if res["decode_tail_frac"].get(cd) and t_dec > t_pre and total in res["decode"]:
                pred[cd] = t_pre + (t_dec - t_pre) * res["decode"][total]["us"] / t_dec
            else:
                pred[cd] = max(t_dec, t_pre)
        res["predicted_step_us"] = {cd: round(v, 2) for cd, v in pred.items()}
        if pred:
            res["predicted_best_cus_decode"] = min(pred, key=pred.get)
    return res


PROFILE_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "profiles")


def profile_from(result):
    """(cus, decode GB/s, prefill TFLOP/s) of a sweep result (dict or JSON file
    path), the alone-phase profile flex_ctl_set_profile takes (Sec. 3.3: the
    scheduler's per-phase profile)."""
    if isinstance(result, str):
        with open(result) as f:
            result = json.load(f)
    cus = sorted(int(c) for c in result["decode"] if str(c) in result["prefill"] or int(c) in result["prefill"])
    get = lambda d, c: d[str(c)] if str(c) in d else d[c]
    return cus, [get(result["decode"], c)["GBps"] for c in cus], [get(result["prefill"], c)["TFLOPs"] for c in cus]


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--workload", default="mixed")
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--pools", type=int, default=4, help="KV cache copies rotated over repetitions")
    ap.add_argument("--cus", default="", help="comma-separated CU counts (default: every eighth of the device)")
    ap.add_argument("--no-corun", action="store_true", help="phase curves only")
    ap.add_argument("--check-outputs", action="store_true", help="co-run vs serial bit-identity at every split")
    ap.add_argument("--save", default="", help="also write the result to this JSON file")
    args = ap.parse_args()
    counts = [int(c) for c in args.cus.split(",") if c] or None
    r = sweep(args.workload, args.reps, args.pools, counts=counts, corun=not args.no_corun,
              check_outputs=args.check_outputs)
    r["command"] = "python -m paper_2606_04415_amd.cusweep " + " ".join(sys.argv[1:])
    if args.save:
        with open(args.save, "w") as f:
            json.dump(r, f, indent=1)
    print(json.dumps(r), flush=True)


if __name__ == "__main__":
    main()
