#!/usr/bin/env python3
"""Benchmark one mixed prefill/decode attention step on one MI355X.

A step is one pass of the whole path over one synthetic batch: the plan
(built once, outside the timed region, like the paper's off-path policy
plane), the prefill kernel and the decode kernel with its split merge, run
either co-located on two CU-masked streams (the default, the paper's dynamic
co-location analog) or serially; a third leg times the one-launch form, in
which one grid holds both phases' work-groups (fused_us). Inputs are
resident in HBM before timing;
the KV cache is rotated over several copies so the 256 MB Infinity Cache
cannot serve repeated steps.

Default workload: the Qwen2.5-7B-shaped mixed step (one 2048-token chunk on
4096 cached tokens plus 128 decodes with context U[1024, 8192], GQA 28/4,
head_dim 128, page 16). Prints one JSON line on stdout.

Each mode runs W warm-up steps, K timed steps (the step time: HIP events on
the issuing stream around the K steps), then K more steps with HIP events
around each phase's kernel on the stream it runs on (the phase durations and
the roofline's kernel duration), kept apart because recording those events
adds about 10 us to a step.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

METRIC = "decode attn HBM GB/s, prefill attn TFLOP/s, mixed-batch step µs (Qwen2.5-7B)"
HBM_PEAK_GBPS = 8000.0
BF16_PEAK_TFLOPS = 2516.6   # 256 CUs x 2.4 GHz x 4096 dense bf16 flop/clk


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def cpu_baseline(b, seconds_target=15.0):
    """Time the fp64 oracle on a bounded sample of the batch; scale to one step."""
    import numpy as np
    import oracle.attention as OA
    w = b.workload
    qsl = b.query_start_loc.tolist()
    ls = b.seq_lens.tolist()
    dec = [s for s in range(len(ls)) if qsl[s + 1] - qsl[s] == 1]
    pre = [s for s in range(len(ls)) if qsl[s + 1] - qsl[s] >= 2]
    kw = dict(num_kv_heads=w.num_kv_heads, page_size=w.page_size, head_dim_v=w.head_dim_v,
              v_aliases_k=w.v_aliases_k)
    t_dec = t_pre = 0.0
    keys_dec_sample = keys_pre_sample = 0
    n_dec_sample = n_pre_rows = 0
    # decode: whole sequences, in batch order, until about half the time budget
    t0 = time.perf_counter()
    for s in dec:
        OA.attention_rows(b.q, b.k_cache, b.v_cache, b.block_table, b.seq_lens, b.query_start_loc,
                          w.sm_scale, [(s, 0)], **kw)
        keys_dec_sample += ls[s]
        n_dec_sample += 1
        if time.perf_counter() - t0 > seconds_target / 2:
            break
    t_dec = time.perf_counter() - t0
    # prefill: groups of 32 rows spread evenly over each chunk, all heads,
    # until the rest of the time budget is spent
    t0 = time.perf_counter()
    budget = max(seconds_target / 2, seconds_target - t_dec)
    for s in pre:
        n, L = qsl[s + 1] - qsl[s], ls[s]
        stride = max(1, n // 32)
        ts = time.perf_counter()
        for off in range(stride):
            rows = list(range(off, n, stride))
            OA.attention_rows(b.q, b.k_cache, b.v_cache, b.block_table, b.seq_lens, b.query_start_loc,
                              w.sm_scale, [(s, i) for i in rows], **kw)
            keys_pre_sample += sum(L - n + i + 1 for i in rows)
            n_pre_rows += len(rows)
            if time.perf_counter() - ts > budget / max(1, len(pre)):
                break
    t_pre = time.perf_counter() - t0
    keys_dec_all = sum(ls[s] for s in dec)
    keys_pre_all = sum(sum(ls[s] - (qsl[s + 1] - qsl[s]) + i + 1 for i in range(qsl[s + 1] - qsl[s])) for s in pre)
    est = 0.0
    if keys_dec_sample:
        est += t_dec * keys_dec_all / keys_dec_sample
    if keys_pre_sample:
        est += t_pre * keys_pre_all / keys_pre_sample
    try:
        from threadpoolctl import threadpool_info
        cores = max([1] + [int(i.get("num_threads", 1)) for i in threadpool_info()])
    except Exception:
        cores = os.cpu_count() or 1
    return {"value": est * 1e6, "unit": "us", "cores": cores, "kind": "oracle",
            "sample": f"{n_dec_sample} of {len(dec)} decode sequences ({keys_dec_sample} keys) + "
                      f"{n_pre_rows} prefill query rows x {w.num_q_heads} heads ({keys_pre_sample} causal keys); "
                      f"{t_dec + t_pre:.1f} s of fp64 numpy, scaled by causal key count to the whole step",
            "measured_s": t_dec + t_pre}


TRAFFIC_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic.json")
KERNEL_SOURCE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2606_04415_amd", "csrc",
                             "attention.hip")


def kernel_source_hash():
    import hashlib
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(workload, kernel):
    """HBM bytes per launch from the committed counter summary, or None when
    there is none for this workload/kernel or the kernels changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    e = t.get("entries", {}).get(f"{workload}:{kernel}")
    return None if e is None else e.get("hbm_bytes_per_launch")


def copy_calibration(nbytes=1 << 30, reps=5):
    """Plain device-to-device copies of a known size, to scale FETCH_SIZE /
    WRITE_SIZE counter readings to bytes."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_launch": nbytes, "launches": reps}), flush=True)


def time_kv_append(b, kv, shape, steps, stream):
    """The step's new tokens appended to the paged pool (not part of `value`):
    average time per append and its HBM rate (rows read once, written once)."""
    import torch
    from paper_2606_04415_amd import flexattn as F
    from paper_2606_04415_amd.workloads import make_append
    a = make_append(b, seed=1)
    dev = torch.device("cuda:0")
    k_new = a.k_new.to(dev)
    v_new = a.v_new.to(dev) if a.v_new is not None else None
    sm = a.slot_mapping.to(dev)
    args = [F.make_append_args(k_new, v_new, sm, k, v) for k, v in kv]
    for i in range(3):
        F.flex_attn_kv_append(shape, args[i % len(args)], stream=stream.cuda_stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(steps):
        F.flex_attn_kv_append(shape, args[i % len(args)], stream=stream.cuda_stream)
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / steps * 1e3
    nbytes = 2 * (k_new.numel() + (v_new.numel() if v_new is not None else 0)) * 2
    return {"tokens": int(sm.numel()), "us": round(us, 2), "GBps": round(nbytes / (us * 1e-6) / 1e9, 1)}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=200,
                    help="untimed steps first: the first passes over the rotated KV copies pay for TLB and clock warm-up")
    ap.add_argument("--workload", default="mixed")
    ap.add_argument("--split", default="128:128", help="prefill:decode CUs for co-run")
    ap.add_argument("--pools", type=int, default=4, help="KV cache copies rotated over steps")
    ap.add_argument("--bm", type=int, default=0, help="prefill rows per tile (0: library default)")
    ap.add_argument("--no-serial", action="store_true", help="skip the serial comparison leg")
    ap.add_argument("--no-fused", action="store_true", help="skip the one-launch (fused) comparison leg")
    ap.add_argument("--fused-wg-per-cu", type=int, default=2,
                    help="decode work-groups per CU the fused leg's plan partitions for")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run plain copies of known size (for scaling memory counters)")
    ap.add_argument("--fused-pass", action="store_true",
                    help="issue warmup + steps one-launch (fused) steps untimed and exit (for kernel tracing)")
    ap.add_argument("--counter-pass", action="store_true",
                    help="only issue the co-run plan's phases one after the other, untimed: the launches a "
                         "co-run step makes, for counter collection (which serialises dispatches and so "
                         "cannot pass the co-run streams' value waits)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: this path has no multi-GPU component "
              "(sequences shard across GPUs with no exchange between them)", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration()
        return

    import torch
    from paper_2606_04415_amd import flexattn as F
    from paper_2606_04415_amd.workloads import WORKLOADS, algorithmic_work, make_batch

    w = WORKLOADS[args.workload]
    log(f"drawing workload '{w.name}': {w.description}")
    b = make_batch(w, seed=0, poison=False)
    ns, ls = b.extra["ns"], b.extra["ls"]
    work = algorithmic_work(w, ns, ls)
    dev = torch.device("cuda:0")
    q = b.q.to(dev)
    kv = []
    for i in range(max(1, args.pools)):
        k = b.k_cache.to(dev)
        v = b.v_cache.to(dev) if b.v_cache is not None else None
        kv.append((k, v))
    bt = b.block_table.to(dev)
    sl = b.seq_lens.to(dev)
    qsl = b.query_start_loc.to(dev)

    cp, cd = (int(x) for x in args.split.split(":"))
    shape = F.make_shape(w.num_q_heads, w.num_kv_heads, w.head_dim_qk, w.head_dim_v, w.page_size,
                         w.sm_scale, w.v_aliases_k)
    t0 = time.perf_counter()
    pa = F.PagedAttention(shape, F.make_opts(cus_decode=cd, bm=args.bm), b.query_start_loc.tolist(), b.seq_lens.tolist(),
                          b.block_table.shape[1])
    plan_us = (time.perf_counter() - t0) * 1e6
    info = pa.plan.info
    out, lse = pa.alloc_out(q)
    arglist = [pa.args(q, k, v, bt, sl, qsl, out) for k, v in kv]
    corun = F.Corun(cp, cd)
    log(f"plan: {info['n_decode_items']} decode items x {info['decode_wg_width']}, "
        f"{info['n_prefill_items']} prefill tiles x {info['prefill_grid_y']}; co-run {cp}/{cd} CUs")

    # The caller issues steps on a stream of its own: HIP's legacy default
    # stream synchronizes implicitly with the co-run pair's streams, which
    # would hold the host at every step.
    caller = torch.cuda.Stream()

    def timed(mode, steps, warmup):
        """K timed steps with nothing but the step in the stream (the step time),
        then K more with HIP events around each phase's kernel on the stream it
        runs on (the phase and kernel durations): recording those events costs
        about 10 us per step, so they stay out of the step time."""
        corun.set_timing(False)
        for i in range(warmup):
            F.flex_attn_mixed(pa.plan, arglist[i % len(arglist)], mode, stream=caller.cuda_stream, corun=corun)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t_wall = time.perf_counter()
        e0.record(caller)
        for i in range(steps):
            F.flex_attn_mixed(pa.plan, arglist[i % len(arglist)], mode, stream=caller.cuda_stream, corun=corun)
        e1.record(caller)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t_wall
        ms = e0.elapsed_time(e1) / steps
        corun.set_timing(True)
        for i in range(steps):
            F.flex_attn_mixed(pa.plan, arglist[i % len(arglist)], mode, stream=caller.cuda_stream, corun=corun)
        torch.cuda.synchronize()
        pre, dec = corun.timing_read()
        corun.set_timing(False)
        return ms, wall, sum(pre) / len(pre), sum(dec) / len(dec)

    if args.counter_pass:
        for i in range(args.warmup + args.steps):
            F.flex_attn_mixed(pa.plan, arglist[i % len(arglist)], F.FLEX_MODE_SERIAL, stream=caller.cuda_stream)
        torch.cuda.synchronize()
        corun.close()
        print(json.dumps({"counter_pass": True, "steps": args.warmup + args.steps, "cus_decode_plan": cd}), flush=True)
        return

    if args.fused_pass:
        pa_f = F.PagedAttention(shape, F.make_opts(cus_decode=0, bm=args.bm, wg_per_cu=args.fused_wg_per_cu),
                                b.query_start_loc.tolist(), b.seq_lens.tolist(), b.block_table.shape[1])
        fargs = [pa_f.args(q, k, v, bt, sl, qsl, out) for k, v in kv]
        for i in range(args.warmup + args.steps):
            F.flex_attn_mixed(pa_f.plan, fargs[i % len(fargs)], F.FLEX_MODE_FUSED, stream=caller.cuda_stream)
        torch.cuda.synchronize()
        corun.close()
        print(json.dumps({"fused_pass": True, "steps": args.warmup + args.steps,
                          "fused_wgs": pa_f.plan.info["n_fused_wgs"]}), flush=True)
        return

    log(f"co-run: {args.warmup} warmup + {args.steps} timed steps")
    c_ms, c_wall, c_pre, c_dec = timed(F.FLEX_MODE_CORUN, args.steps, args.warmup)
    log(f"co-run step {c_ms * 1e3:.1f} us (prefill {c_pre * 1e3:.1f} us, decode {c_dec * 1e3:.1f} us)")
    s_ms = s_pre = s_dec = None
    if not args.no_serial:
        # serial leg: the same batch planned for the whole device
        pa_s = F.PagedAttention(shape, F.make_opts(cus_decode=0, bm=args.bm), b.query_start_loc.tolist(),
                                b.seq_lens.tolist(), b.block_table.shape[1])
        arglist = [pa_s.args(q, k, v, bt, sl, qsl, out) for k, v in kv]
        pa = pa_s
        s_ms, _, s_pre, s_dec = timed(F.FLEX_MODE_SERIAL, args.steps, args.warmup)
        log(f"serial step {s_ms * 1e3:.1f} us (prefill {s_pre * 1e3:.1f} us, decode {s_dec * 1e3:.1f} us)")
    corun.close()
    f_ms = None
    if not args.no_fused:
        # fused leg: both phases in one launch, the work-groups interleaved by the plan
        pa_f = F.PagedAttention(shape, F.make_opts(cus_decode=0, bm=args.bm, wg_per_cu=args.fused_wg_per_cu),
                                b.query_start_loc.tolist(), b.seq_lens.tolist(), b.block_table.shape[1])
        if pa_f.plan.info["n_fused_wgs"] > 0:
            fargs = [pa_f.args(q, k, v, bt, sl, qsl, out) for k, v in kv]
            for i in range(args.warmup):
                F.flex_attn_mixed(pa_f.plan, fargs[i % len(fargs)], F.FLEX_MODE_FUSED, stream=caller.cuda_stream)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(caller)
            for i in range(args.steps):
                F.flex_attn_mixed(pa_f.plan, fargs[i % len(fargs)], F.FLEX_MODE_FUSED, stream=caller.cuda_stream)
            e1.record(caller)
            torch.cuda.synchronize()
            f_ms = e0.elapsed_time(e1) / args.steps
            log(f"fused step {f_ms * 1e3:.1f} us ({pa_f.plan.info['n_fused_wgs']} work-groups)")

    dec_bytes = work["decode"]["bytes"]
    pre_flops = work["prefill"]["flops"]
    # dominant kernel: the one with the larger share of the co-run step;
    # frac_of_cu_share prices it against the peak of the CUs its stream holds
    n_cus = torch.cuda.get_device_properties(0).multi_processor_count
    if dec_bytes and (not pre_flops or c_dec >= c_pre):
        achieved = dec_bytes / (c_dec * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": measured_traffic(w.name, "decode"),
                "kernel": "decode_gqa_kernel" if w.head_dim_qk != 576 else "rowpar_kernel (latent decode)",
                "algorithmic_bytes_per_launch": dec_bytes, "avg_launch_us": round(c_dec * 1e3, 2),
                "cus": cd}
    else:
        achieved = pre_flops / (c_pre * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": measured_traffic(w.name, "prefill"),
                "kernel": "rowpar_kernel (prefill)", "algorithmic_flops_per_launch": pre_flops,
                "avg_launch_us": round(c_pre * 1e3, 2), "cus": cp,
                "frac_of_cu_share": round(achieved / (BF16_PEAK_TFLOPS * cp / n_cus), 4)}

    result = {
        "metric": METRIC, "value": round(c_ms * 1e3, 2), "unit": "us", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(c_ms, 5), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.description}", "batch": len(ls), "query_tokens": sum(ns),
                   "kv_tokens": sum(ls), "mode": "corun", "cus_prefill": cp, "cus_decode": cd,
                   "kv_pools": len(kv), "plan_host_us": round(plan_us, 1)},
        "phases_us": {"corun_prefill": round(c_pre * 1e3, 2), "corun_decode": round(c_dec * 1e3, 2)},
        "roofline": roof,
    }
    # the other phase of the co-run step against its own peak (HBM is shared
    # by the whole device, so a bandwidth-bound phase is priced against all of it)
    if dec_bytes and pre_flops:
        if roof["bound"] == "mfma":
            a = dec_bytes / (c_dec * 1e-3) / 1e9
            result["roofline_other"] = {"bound": "hbm", "kernel": "decode_gqa_kernel + merge_kernel",
                                        "achieved": round(a, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                        "frac": round(a / HBM_PEAK_GBPS, 4), "cus": cd,
                                        "avg_phase_us": round(c_dec * 1e3, 2)}
        else:
            a = pre_flops / (c_pre * 1e-3) / 1e12
            result["roofline_other"] = {"bound": "mfma", "kernel": "rowpar_kernel (prefill)",
                                        "achieved": round(a, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                        "frac": round(a / BF16_PEAK_TFLOPS, 4), "cus": cp,
                                        "frac_of_cu_share": round(a / (BF16_PEAK_TFLOPS * cp / n_cus), 4),
                                        "avg_phase_us": round(c_pre * 1e3, 2)}
    if s_ms is not None:
        result["serial_us"] = round(s_ms * 1e3, 2)
        result["corun_speedup_vs_serial"] = round(s_ms / c_ms, 4)
        result["phases_us"].update({"serial_prefill": round(s_pre * 1e3, 2), "serial_decode": round(s_dec * 1e3, 2)})
        if dec_bytes:
            result["decode_GBps_all_cus"] = round(dec_bytes / (s_dec * 1e-3) / 1e9, 1)
        if pre_flops:
            result["prefill_TFLOPs_all_cus"] = round(pre_flops / (s_pre * 1e-3) / 1e12, 2)
    if f_ms is not None:
        result["fused_us"] = round(f_ms * 1e3, 2)
        result["fused_wg_per_cu"] = args.fused_wg_per_cu
        if s_ms is not None:
            result["fused_speedup_vs_serial"] = round(s_ms / f_ms, 4)
    result["bound_us"] = round(max((dec_bytes + work["prefill"]["bytes"]) / (HBM_PEAK_GBPS * 1e3),
                                   (pre_flops + work["decode"]["flops"]) / (BF16_PEAK_TFLOPS * 1e6)), 1)
    result["kv_append"] = time_kv_append(b, kv, shape, args.steps, caller)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline(b, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
