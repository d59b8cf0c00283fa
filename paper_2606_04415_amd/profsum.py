"""Summarise rocprofv3 CSV output of bench.py runs into the committed profile files.

Kernel statistics (``--kernel-trace --stats``) become a markdown table;
per-dispatch FETCH_SIZE / WRITE_SIZE counters (``--pmc``), scaled by what the
same counters read for a device copy of known size (``bench.py
--copy-calibration``), become HBM bytes per launch in ``traffic.json``, keyed
to the kernel source they were measured on (bench.py drops them once the
kernels change).

    python -m paper_2606_04415_amd.profsum stats <kernel_stats.csv> <title> <command> > profiles/x.md
    python -m paper_2606_04415_amd.profsum traffic --workload mixed --fetch <csv> --write <csv> \\
        --copy-fetch <csv> --copy-write <csv> --command "..." [--command "..."] [--into traffic.json] > new.json
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import sys
from collections import defaultdict

KERNEL_SOURCE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "attention.hip")
COPY_BYTES = 1 << 30


def code_text(src: str) -> str:
    """The kernel source with its comments and whitespace removed: edits of
    comments leave what is measured unchanged."""
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def source_hash(path: str = KERNEL_SOURCE) -> str:
    with open(path, encoding="utf-8") as f:
        return hashlib.sha256(code_text(f.read()).encode()).hexdigest()[:16]


def stats_table(path, title, command):
    rows = list(csv.DictReader(open(path)))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    out = [f"# {title}", "", "Command (repository root, one MI355X):", "", f"    {command}", "",
           "| kernel | calls | avg us | min us | max us | share |", "|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| `{r['Name'][:90]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                   f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                   f"{float(r['TotalDurationNs']) / total * 100:.1f}% |")
    return "\n".join(out) + "\n"


def kernel_role(name):
    """decode / prefill / merge for the library's kernels, None for others.
    rowpar_kernel's seventh template argument is its row layout (2: latent
    decode rows, else prefill tiles)."""
    if "merge_kernel" in name:
        return "merge"
    if "decode_gqa_kernel" in name:
        return "decode"
    if "flat_prefill_kernel" in name:
        return "prefill"
    if "rowpar_kernel<" in name:
        targs = name.split("rowpar_kernel<", 1)[1].split(">", 1)[0].split(",")
        return "decode" if len(targs) > 6 and targs[6].strip() == "2" else "prefill"
    return None


def counter_means(path, counter):
    """Mean per-dispatch value of `counter` for each kernel name (KiB for the size counters)."""
    acc, n = defaultdict(float), defaultdict(set)
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        acc[r["Kernel_Name"]] += float(r["Counter_Value"])
        n[r["Kernel_Name"]].add(r["Dispatch_Id"])
    return {k: acc[k] / len(n[k]) for k in acc}


def traffic(args):
    cf = counter_means(args.copy_fetch, "FETCH_SIZE")
    cw = counter_means(args.copy_write, "WRITE_SIZE")
    copy_kernel = max(cf, key=cf.get)
    fetch_scale = COPY_BYTES / 1024 / cf[copy_kernel]
    write_scale = COPY_BYTES / 1024 / cw[max(cw, key=cw.get)]
    f = counter_means(args.fetch, "FETCH_SIZE")
    w = counter_means(args.write, "WRITE_SIZE")
    entries = {}
    if args.into and os.path.exists(args.into):
        with open(args.into) as fh:
            prev = json.load(fh)
        if prev.get("kernel_source_sha256_16") == source_hash():
            entries.update(prev.get("entries", {}))
            args.command = prev.get("commands", []) + [c for c in args.command if c not in prev.get("commands", [])]
    for name in f:
        role = kernel_role(name)
        if role is None:
            continue
        fb = f[name] * 1024 * fetch_scale
        wb = w.get(name, 0.0) * 1024 * write_scale
        entries[f"{args.workload}:{role}"] = {
            "kernel": name, "fetch_kib_raw": round(f[name], 1), "write_kib_raw": round(w.get(name, 0.0), 1),
            "hbm_bytes_per_launch": int(fb + wb), "fetch_bytes": int(fb), "write_bytes": int(wb)}
    return {"kernel_source_sha256_16": source_hash(), "fetch_scale": fetch_scale, "write_scale": write_scale,
            "calibration": f"1 GiB device copy (bench.py --copy-calibration): FETCH_SIZE {cf[copy_kernel]:.0f} KiB, "
                           f"WRITE_SIZE {cw[max(cw, key=cw.get)]:.0f} KiB per launch",
            "commands": args.command, "entries": entries}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("title")
    s.add_argument("command")
    t = sub.add_parser("traffic")
    t.add_argument("--workload", default="mixed")
    for k in ("fetch", "write", "copy_fetch", "copy_write"):
        t.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    t.add_argument("--command", action="append", default=[])
    t.add_argument("--into", default="",
                   help="an existing traffic.json whose entries (same kernel source) are kept")
    a = ap.parse_args()
    if a.cmd == "stats":
        sys.stdout.write(stats_table(a.csv, a.title, a.command))
    else:
        print(json.dumps(traffic(a), indent=1))


if __name__ == "__main__":
    main()
