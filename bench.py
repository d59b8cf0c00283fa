#!/usr/bin/env python3
"""Benchmark one mixed prefill/decode attention step on one MI355X, plus the
single-phase workloads, each against its roofline.

A step is one pass of the whole path over one synthetic batch: the plan
(built once, outside the timed region, like the paper's off-path policy
plane), the prefill kernel and the decode kernel with its split merge, run
co-located on two CU-masked streams (the headline, the paper's dynamic
co-location analog; 160 prefill / 96 decode CUs by default, the decode
ranges that remain when the prefill ends running on the prefill share as the
plan's decode tail), serially on one stream, or as one launch holding both
phases' work-groups. Inputs are resident in HBM before timing; KV caches
that the 256 MB Infinity Cache could hold are rotated over several copies.

Headline workload: the Qwen2.5-7B-shaped mixed step (one 2048-token chunk on
4096 cached tokens plus 128 decodes with context U[1024, 8192], GQA 28/4,
head_dim 128, page 16). Also timed: the 64-sequence decode batch (decode
GB/s), the 8 x 2048 causal prefill (prefill TFLOP/s) and the absorbed-MLA
step (decode, prefill, serial step). Prints one JSON line on stdout.

Protocol. The device raises its clock over the first ~100-200 MFMA-heavy
launches after it has been idle (prefill 219 -> 181 us; again after one
second idle); decode is flat. So the setup runs untimed steps of every leg
until about `--settle-ms` of work has passed ("settle" in the line), after
the W warm-up steps; the K co-run steps right after the warm-up, before the
settle, are reported as `cold_corun_us`. The legs are then timed
interleaved: blocks of steps of each mode in rotating order, each block
bracketed by synchronisations and one pair of HIP events; `value` is the
co-run blocks' time over K and every leg's `mean` comes from its blocks.
Recording an event between steps adds work to the stream (about 3 us per
decode step, 5 us per co-run step), so the p10/p50/p90 of each leg come from
a separate pass with an event after every step, whose mean is reported as
`per_step_events_mean`. A further pass with HIP events around each phase's
kernels (on the stream they run on) gives the phase durations for the
roofline. Last, the fixed half-and-half split (128 / 128 CUs, its plan's
own decode tail) runs on a co-run pair of its own, timed the same way
(`corun_half_split`), beside the chosen split and the serial step.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

METRIC = "decode attn HBM GB/s, prefill attn TFLOP/s, mixed-batch step µs (Qwen2.5-7B)"
HBM_PEAK_GBPS = 8000.0
BF16_PEAK_TFLOPS = 2516.6   # 256 CUs x 2.4 GHz x 4096 dense bf16 flop/clk


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def pct(xs, q):
    ys = sorted(xs)
    if not ys:
        return None
    k = (len(ys) - 1) * q
    lo, hi = math.floor(k), math.ceil(k)
    return ys[lo] + (ys[hi] - ys[lo]) * (k - lo)


def dist(us):
    return {"mean": round(sum(us) / len(us), 2), "p10": round(pct(us, 0.1), 2), "p50": round(pct(us, 0.5), 2),
            "p90": round(pct(us, 0.9), 2), "n": len(us)}


def host_info():
    info = {"cpu_count": os.cpu_count()}
    try:
        info["affinity"] = len(os.sched_getaffinity(0))
    except Exception:
        info["affinity"] = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    info["cpu_model"] = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        info["blas_threads"] = max([1] + [int(i.get("num_threads", 1)) for i in threadpool_info()])
    except Exception:
        info["blas_threads"] = None
    return info


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
    hi = host_info()
    cores = hi.get("blas_threads") or hi.get("affinity") or os.cpu_count() or 1
    return {"value": est * 1e6, "unit": "us", "cores": cores, "kind": "oracle", "host": hi,
            "sample": f"{n_dec_sample} of {len(dec)} decode sequences ({keys_dec_sample} keys) + "
                      f"{n_pre_rows} prefill query rows x {w.num_q_heads} heads ({keys_pre_sample} causal keys); "
                      f"{t_dec + t_pre:.1f} s of fp64 numpy, scaled by causal key count to the whole step",
            "measured_s": t_dec + t_pre}


TRAFFIC_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic.json")
KERNEL_SOURCE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2606_04415_amd", "csrc",
                             "attention.hip")


def kernel_source_hash():
    """Hash of the kernel source's code (comments and whitespace removed),
    the key of the committed counter summary."""
    from paper_2606_04415_amd.profsum import source_hash
    return source_hash(KERNEL_SOURCE)


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


def launch_timer(stream, fn, n, settle_ms, warmup):
    """Settle, then time n launches back to back between one pair of events
    (their mean, us), and n more with an event after each (per-launch us,
    for the distribution; the events add work to the stream). Returns
    (mean, per-launch list, settle launches)."""
    import torch
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    i = 0
    while time.perf_counter() - t0 < settle_ms * 1e-3:
        for _ in range(10):
            fn(i)
            i += 1
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for j in range(n):
        fn(j)
    e1.record(stream)
    torch.cuda.synchronize()
    mean = e0.elapsed_time(e1) * 1e3 / n
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    ev[0].record(stream)
    for j in range(n):
        fn(j)
        ev[j + 1].record(stream)
    torch.cuda.synchronize()
    return mean, [ev[j].elapsed_time(ev[j + 1]) * 1e3 for j in range(n)], i


def timed_dist(mean, per):
    """mean from an unbroken block; p10/p50/p90 from the per-step pass."""
    d = dist(per)
    d["per_step_events_mean"] = d["mean"]
    d["mean"] = round(mean, 2)
    return d


def prefill_kernel_name(bm, head_dim_qk):
    """The kernel a plan's prefill tiles run on."""
    if head_dim_qk in (64, 128) and bm == 128:
        return "flat_prefill_kernel"
    return "rowpar_kernel (prefill)"


def roof(bound, achieved, unit):
    peak = HBM_PEAK_GBPS if bound == "hbm" else BF16_PEAK_TFLOPS
    return {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit, "frac": round(achieved / peak, 4)}


def bench_config(name, steps, warmup, settle_ms, pools):
    """Single-phase workloads and the latent step, on all CUs, plans with
    library defaults; per-launch times and roofline fractions."""
    import torch
    from paper_2606_04415_amd import flexattn as F
    from paper_2606_04415_amd.workloads import WORKLOADS, algorithmic_work, make_batch
    w = WORKLOADS[name]
    b = make_batch(w, seed=0, poison=False, device="cuda")
    work = algorithmic_work(w, b.extra["ns"], b.extra["ls"])
    dev = torch.device("cuda:0")
    kv = [(b.k_cache, b.v_cache)] + [(b.k_cache.clone(), None if b.v_cache is None else b.v_cache.clone())
                                     for _ in range(pools - 1)]
    bt, sl, qsl = b.block_table.to(dev), b.seq_lens.to(dev), b.query_start_loc.to(dev)
    shape = F.make_shape(w.num_q_heads, w.num_kv_heads, w.head_dim_qk, w.head_dim_v, w.page_size,
                         w.sm_scale, w.v_aliases_k)
    pa = F.PagedAttention(shape, None, b.query_start_loc.tolist(), b.seq_lens.tolist(), b.block_table.shape[1])
    out, _ = pa.alloc_out(b.q)
    args = [pa.args(b.q, k, v, bt, sl, qsl, out) for k, v in kv]
    st = torch.cuda.Stream()
    cs = st.cuda_stream
    res = {"workload": f"{w.name}: {w.description}", "kv_pools": pools, "bm": pa.plan.info["bm"],
           "inputs": "q/k/v drawn on the device (seeded), ~N(0,1) in bf16"}
    dec_b, pre_f = work["decode"]["bytes"], work["prefill"]["flops"]
    legs = []
    if dec_b:
        legs.append(("decode", lambda i: F.flex_attn_decode(pa.plan, args[i % len(args)], stream=cs)))
    if pre_f:
        legs.append(("prefill", lambda i: F.flex_attn_prefill(pa.plan, args[i % len(args)], stream=cs)))
    if dec_b and pre_f:
        legs.append(("serial_step", lambda i: F.flex_attn_mixed(pa.plan, args[i % len(args)], F.FLEX_MODE_SERIAL,
                                                                stream=cs)))
    for leg, fn in legs:
        mean, us, settled = launch_timer(st, fn, steps, settle_ms, warmup)
        d = timed_dist(mean, us)
        r = {"us": d, "settle_launches": settled}
        if leg == "decode":
            r["GBps"] = round(dec_b / (d["mean"] * 1e-6) / 1e9, 1)
            r["roofline"] = roof("hbm", r["GBps"], "GB/s")
            r["roofline"]["traffic"] = measured_traffic(name, "decode")
            r["kernel"] = "decode_gqa_kernel + merge_kernel" if w.head_dim_qk != 576 else \
                "rowpar_kernel (latent decode) + merge_kernel"
            r["algorithmic_bytes"] = dec_b
            if w.head_dim_qk == 576:   # latent decode sits near the ridge: its MFMA side too
                fl = work["decode"]["flops"]
                r["TFLOPs"] = round(fl / (d["mean"] * 1e-6) / 1e12, 1)
                r["bound_us"] = round(max(dec_b / (HBM_PEAK_GBPS * 1e3), fl / (BF16_PEAK_TFLOPS * 1e6)), 1)
        elif leg == "prefill":
            r["TFLOPs"] = round(pre_f / (d["mean"] * 1e-6) / 1e12, 1)
            r["roofline"] = roof("mfma", r["TFLOPs"], "TFLOP/s")
            r["roofline"]["traffic"] = measured_traffic(name, "prefill")
            r["kernel"] = prefill_kernel_name(pa.plan.info["bm"], w.head_dim_qk)
            r["algorithmic_flops"] = pre_f
        else:
            r["bound_us"] = round(max((dec_b + work["prefill"]["bytes"]) / (HBM_PEAK_GBPS * 1e3),
                                      (pre_f + work["decode"]["flops"]) / (BF16_PEAK_TFLOPS * 1e6)), 1)
            r["frac_of_bound"] = round(r["bound_us"] / d["mean"], 4)
        res[leg] = r
        log(f"{name} {leg}: {d['mean']:.1f} us (p10 {d['p10']:.1f}, p90 {d['p90']:.1f})")
    del kv, args, b
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--settle-ms", type=float, default=400.0,
                    help="untimed steps of every leg after the warm-up, until this much time has passed")
    ap.add_argument("--workload", default="mixed")
    ap.add_argument("--split", default="160:96", help="prefill:decode CUs for co-run")
    ap.add_argument("--pools", type=int, default=4, help="KV cache copies rotated over steps")
    ap.add_argument("--bm", type=int, default=0, help="prefill rows per tile (0: library default)")
    ap.add_argument("--blocks", type=int, default=5, help="interleaved timing blocks per leg")
    ap.add_argument("--no-serial", action="store_true", help="skip the serial comparison leg")
    ap.add_argument("--no-half", action="store_true", help="skip the fixed half-and-half co-run split")
    ap.add_argument("--no-fused", action="store_true", help="skip the one-launch (fused) comparison leg")
    ap.add_argument("--no-configs", action="store_true", help="skip the single-phase and latent workloads")
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
    ap.add_argument("--config-pass", default="",
                    help="only issue warmup + steps serial steps of this workload (library defaults), untimed "
                         "(for kernel tracing and counters of the single-phase and latent workloads)")
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

    if args.config_pass:
        w = WORKLOADS[args.config_pass]
        b = make_batch(w, seed=0, poison=False, device="cuda")
        dev = torch.device("cuda:0")
        bt, sl, qsl = b.block_table.to(dev), b.seq_lens.to(dev), b.query_start_loc.to(dev)
        shape = F.make_shape(w.num_q_heads, w.num_kv_heads, w.head_dim_qk, w.head_dim_v, w.page_size,
                             w.sm_scale, w.v_aliases_k)
        pa = F.PagedAttention(shape, F.make_opts(bm=args.bm), b.query_start_loc.tolist(), b.seq_lens.tolist(),
                              b.block_table.shape[1])
        out, _ = pa.alloc_out(b.q)
        a = pa.args(b.q, b.k_cache, b.v_cache, bt, sl, qsl, out)
        for i in range(args.warmup + args.steps):
            F.flex_attn_mixed(pa.plan, a, F.FLEX_MODE_SERIAL)
        torch.cuda.synchronize()
        print(json.dumps({"config_pass": args.config_pass, "steps": args.warmup + args.steps,
                          "bm": pa.plan.info["bm"]}), flush=True)
        return

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
    plan_us = []
    def plan(**kw):
        t0 = time.perf_counter()
        pa = F.PagedAttention(shape, F.make_opts(bm=args.bm, **kw), b.query_start_loc.tolist(), b.seq_lens.tolist(),
                              b.block_table.shape[1])
        plan_us.append((time.perf_counter() - t0) * 1e6)
        return pa
    pa_c = plan(cus_decode=cd)
    pa_s = plan(cus_decode=0)
    pa_f = plan(cus_decode=0, wg_per_cu=args.fused_wg_per_cu)
    out, lse = pa_c.alloc_out(q)
    arg_c = [pa_c.args(q, k, v, bt, sl, qsl, out) for k, v in kv]
    arg_s = [pa_s.args(q, k, v, bt, sl, qsl, out) for k, v in kv]
    arg_f = [pa_f.args(q, k, v, bt, sl, qsl, out) for k, v in kv]
    corun = F.Corun(cp, cd)
    info = pa_c.plan.info
    log(f"plan: {info['n_decode_items']} decode items x {info['decode_wg_width']}, "
        f"{info['n_prefill_items']} prefill tiles x {info['prefill_grid_y']} (bm {info['bm']}); co-run {cp}/{cd} CUs")

    # The caller issues steps on a stream of its own: HIP's legacy default
    # stream synchronizes implicitly with the co-run pair's streams.
    caller = torch.cuda.Stream()
    cs = caller.cuda_stream
    step = {
        "corun": lambda i: F.flex_attn_mixed(pa_c.plan, arg_c[i % len(arg_c)], F.FLEX_MODE_CORUN, stream=cs,
                                             corun=corun),
        "serial": lambda i: F.flex_attn_mixed(pa_s.plan, arg_s[i % len(arg_s)], F.FLEX_MODE_SERIAL, stream=cs),
        "fused": lambda i: F.flex_attn_mixed(pa_f.plan, arg_f[i % len(arg_f)], F.FLEX_MODE_FUSED, stream=cs),
    }
    legs = ["corun"] + ([] if args.no_serial else ["serial"]) + \
           ([] if args.no_fused or pa_f.plan.info["n_fused_wgs"] == 0 else ["fused"])

    if args.counter_pass:
        for i in range(args.warmup + args.steps):
            F.flex_attn_mixed(pa_c.plan, arg_c[i % len(arg_c)], F.FLEX_MODE_SERIAL, stream=cs)
        torch.cuda.synchronize()
        corun.close()
        print(json.dumps({"counter_pass": True, "steps": args.warmup + args.steps, "cus_decode_plan": cd}), flush=True)
        return
    if args.fused_pass:
        for i in range(args.warmup + args.steps):
            step["fused"](i)
        torch.cuda.synchronize()
        corun.close()
        print(json.dumps({"fused_pass": True, "steps": args.warmup + args.steps,
                          "fused_wgs": pa_f.plan.info["n_fused_wgs"]}), flush=True)
        return

    def block(mode, n, start, per_step=False):
        """n steps of one mode back to back between one pair of events; with
        per_step, an event after every step too. Returns (per-step times or
        [], the block's time), us."""
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
        torch.cuda.synchronize()
        ev[0].record(caller)
        for j in range(n):
            step[mode](start + j)
            if per_step or j == n - 1:
                ev[j + 1].record(caller)
        torch.cuda.synchronize()
        per = [ev[j].elapsed_time(ev[j + 1]) * 1e3 for j in range(n)] if per_step else []
        return per, ev[0].elapsed_time(ev[n]) * 1e3

    # W warm-up steps, then K co-run steps before settling (the cold figure)
    log(f"warm-up: {args.warmup} steps; cold co-run: {args.steps} steps")
    for i in range(args.warmup):
        step["corun"](i)
    _, cold_total = block("corun", args.steps, args.warmup)
    # settle: rotate the legs until settle_ms have passed
    t0 = time.perf_counter()
    n_settle = 0
    while time.perf_counter() - t0 < args.settle_ms * 1e-3:
        for mode in legs:
            for _ in range(5):
                step[mode](n_settle)
                n_settle += 1
        torch.cuda.synchronize()
    settle_ms = (time.perf_counter() - t0) * 1e3
    log(f"settle: {n_settle} steps in {settle_ms:.0f} ms; timing {args.steps} steps per leg in "
        f"{args.blocks} interleaved blocks")
    per = {m: [] for m in legs}
    total = {m: 0.0 for m in legs}
    nb = max(1, min(args.blocks, args.steps))
    sizes = [args.steps // nb + (1 if r < args.steps % nb else 0) for r in range(nb)]
    for r in range(nb):
        order = legs[r % len(legs):] + legs[:r % len(legs)]
        for mode in order:
            _, t = block(mode, sizes[r], r * 1000)
            total[mode] += t
    # the distribution: one more pass per leg with an event after every step
    for mode in legs:
        per[mode], _ = block(mode, args.steps, 9000, per_step=True)
    c_ms = total["corun"] / args.steps / 1e3

    # phase durations (events on each kernel's own stream), a separate pass
    def phases(mode, pa_, arg_):
        corun.set_timing(True)
        for i in range(args.steps):
            F.flex_attn_mixed(pa_.plan, arg_[i % len(arg_)], mode, stream=cs, corun=corun)
        torch.cuda.synchronize()
        pre, dec = corun.timing_read()
        corun.set_timing(False)
        return sum(pre) / len(pre), sum(dec) / len(dec), pre, dec
    c_pre, c_dec, c_pre_l, c_dec_l = phases(F.FLEX_MODE_CORUN, pa_c, arg_c)
    s_pre = s_dec = None
    if "serial" in legs:
        s_pre, s_dec, _, _ = phases(F.FLEX_MODE_SERIAL, pa_s, arg_s)
    corun.close()

    # The fixed half-and-half split beside the chosen one, on a pair of its own
    # opened once the chosen split's pair is closed (pairs open together share
    # the hardware queues); timed after the other legs, on a settled device.
    n_cus = torch.cuda.get_device_properties(0).multi_processor_count
    half = None
    if not args.no_half and cp + cd == n_cus and cd != n_cus // 2:
        pa_h = F.PagedAttention(shape, F.make_opts(bm=args.bm, cus_decode=n_cus // 2), b.query_start_loc.tolist(),
                                b.seq_lens.tolist(), b.block_table.shape[1])
        arg_h = [pa_h.args(q, k, v, bt, sl, qsl, out) for k, v in kv]
        corun_h = F.Corun(n_cus // 2, n_cus // 2)
        step["half"] = lambda i: F.flex_attn_mixed(pa_h.plan, arg_h[i % len(arg_h)], F.FLEX_MODE_CORUN, stream=cs,
                                                   corun=corun_h)
        for i in range(max(100, args.warmup)):   # the new pair's first steps run slower
            step["half"](i)
        _, t_half = block("half", args.steps, 20000)
        per_half, _ = block("half", args.steps, 30000, per_step=True)
        corun_h.close()
        half = {"cus_prefill": n_cus // 2, "cus_decode": n_cus // 2,
                "decode_tail_ranges": pa_h.plan.info["n_decode_tail_ranges"],
                "step_us": timed_dist(t_half / args.steps, per_half)}

    dec_bytes = work["decode"]["bytes"]
    pre_flops = work["prefill"]["flops"]
    # the co-run decode phase (events on the decode stream) streams the decode
    # share's ranges; a decode tail runs on the prefill stream after the prefill
    tail_frac = info["decode_tail_bytes"] / info["decode_bytes"] if info["decode_bytes"] else 0.0
    dec_share_bytes = dec_bytes * (1.0 - tail_frac)
    dec_phase_kernel = "decode_gqa_kernel" + (" (decode share's ranges)" if tail_frac else " + merge_kernel")
    all_traffic = measured_traffic(w.name, "decode")
    share_traffic = None if all_traffic is None else round(all_traffic * (1.0 - tail_frac))
    # dominant kernel: the phase with the larger share of the co-run step
    if dec_bytes and (not pre_flops or c_dec >= c_pre):
        achieved = dec_share_bytes / (c_dec * 1e-3) / 1e9
        roof_ = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                 "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": share_traffic,
                 "kernel": "decode_gqa_kernel" if w.head_dim_qk != 576 else "rowpar_kernel (latent decode)",
                 "algorithmic_bytes_per_launch": round(dec_share_bytes), "avg_launch_us": round(c_dec * 1e3, 2),
                 "cus": cd}
        if tail_frac and share_traffic is not None:
            roof_["traffic_note"] = ("counter bytes of one launch over every decode range (the counter pass), "
                                     "times the decode share's fraction of the algorithmic bytes")
    else:
        achieved = pre_flops / (c_pre * 1e-3) / 1e12
        roof_ = {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                 "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": measured_traffic(w.name, "prefill"),
                 "kernel": prefill_kernel_name(info["bm"], w.head_dim_qk), "algorithmic_flops_per_launch": pre_flops,
                 "avg_launch_us": round(c_pre * 1e3, 2), "cus": cp,
                 "frac_of_cu_share": round(achieved / (BF16_PEAK_TFLOPS * cp / n_cus), 4)}

    result = {
        "metric": METRIC, "value": round(c_ms * 1e3, 2), "unit": "us", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(c_ms, 5), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.description}", "batch": len(ls), "query_tokens": sum(ns),
                   "kv_tokens": sum(ls), "mode": "corun", "cus_prefill": cp, "cus_decode": cd,
                   "kv_pools": len(kv), "prefill_bm": info["bm"], "plan_host_us": [round(x, 1) for x in plan_us],
                   "decode_tail": {"ranges": info["n_decode_tail_ranges"], "of_ranges": info["n_decode_ranges"],
                                   "bytes_frac": round(tail_frac, 4)}},
        "settle": {"steps": n_settle, "ms": round(settle_ms, 1),
                   "why": "untimed steps of every leg after the warm-up: the device raises its clock over the first "
                          "~100-200 MFMA-heavy launches after idle"},
        "cold_corun_us": round(cold_total / args.steps, 2),
        "step_us": {m: timed_dist(total[m] / args.steps, per[m]) for m in legs},
        "phases_us": {"corun_prefill": round(c_pre * 1e3, 2), "corun_decode": round(c_dec * 1e3, 2)},
        "roofline": roof_,
    }
    if dec_bytes and pre_flops:
        if roof_["bound"] == "mfma":
            a = dec_share_bytes / (c_dec * 1e-3) / 1e9
            result["roofline_other"] = {"bound": "hbm", "kernel": dec_phase_kernel,
                                        "achieved": round(a, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                        "frac": round(a / HBM_PEAK_GBPS, 4), "cus": cd,
                                        "avg_phase_us": round(c_dec * 1e3, 2)}
        else:
            a = pre_flops / (c_pre * 1e-3) / 1e12
            result["roofline_other"] = {"bound": "mfma", "kernel": prefill_kernel_name(info["bm"], w.head_dim_qk),
                                        "achieved": round(a, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                        "frac": round(a / BF16_PEAK_TFLOPS, 4), "cus": cp,
                                        "frac_of_cu_share": round(a / (BF16_PEAK_TFLOPS * cp / n_cus), 4),
                                        "avg_phase_us": round(c_pre * 1e3, 2)}
    if "serial" in legs:
        s_ms = total["serial"] / args.steps / 1e3
        result["serial_us"] = round(s_ms * 1e3, 2)
        result["corun_speedup_vs_serial"] = round(s_ms / c_ms, 4)
        result["phases_us"].update({"serial_prefill": round(s_pre * 1e3, 2), "serial_decode": round(s_dec * 1e3, 2)})
        if dec_bytes:
            result["decode_GBps_all_cus"] = round(dec_bytes / (s_dec * 1e-3) / 1e9, 1)
        if pre_flops:
            result["prefill_TFLOPs_all_cus"] = round(pre_flops / (s_pre * 1e-3) / 1e12, 2)
        if half is not None:
            half["speedup_vs_serial"] = round(s_ms * 1e3 / half["step_us"]["mean"], 4)
    if half is not None:
        result["corun_half_split"] = half
    if "fused" in legs:
        f_ms = total["fused"] / args.steps / 1e3
        result["fused_us"] = round(f_ms * 1e3, 2)
        result["fused_wg_per_cu"] = args.fused_wg_per_cu
        if "serial" in legs:
            result["fused_speedup_vs_serial"] = round(total["serial"] / total["fused"], 4)
    result["bound_us"] = round(max((dec_bytes + work["prefill"]["bytes"]) / (HBM_PEAK_GBPS * 1e3),
                                   (pre_flops + work["decode"]["flops"]) / (BF16_PEAK_TFLOPS * 1e6)), 1)
    result["max_phase_us"] = round(max(c_pre, c_dec) * 1e3, 2)
    result["kv_append"] = time_kv_append(b, kv, shape, args.steps, caller)
    del kv, arg_c, arg_s, arg_f, q
    if half is not None:
        del arg_h, pa_h
    torch.cuda.empty_cache()
    if not args.no_configs:
        result["configs"] = {}
        for name, pools in (("decode", 4), ("prefill", 2), ("mla", 1)):
            log(f"workload '{name}'")
            result["configs"][name] = bench_config(name, args.steps, args.warmup, args.settle_ms / 2, pools)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline(b, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
