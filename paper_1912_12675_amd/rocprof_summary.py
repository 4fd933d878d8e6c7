"""Summaries of rocprofv3 output for the kernels of libpsw.

    python -m paper_1912_12675_amd.rocprof_summary stats KERNEL_STATS_CSV --steps N [--top 25]
        per-kernel table (calls per step, mean / total time) of a
        `rocprofv3 --kernel-trace --stats --output-format csv` run

    python -m paper_1912_12675_amd.rocprof_summary traffic --kernel NAME [--kernel NAME ...] \
            --fetch PMC_CSV --write PMC_CSV --copy-fetch PMC_CSV --copy-write PMC_CSV \
            --copy-kernel SUBSTRING --copy-bytes B [--out profiles/traffic.json]
        HBM bytes per launch of each kernel NAME from two `--pmc FETCH_SIZE`
        and `--pmc WRITE_SIZE` runs, each counter scaled by what it reads for
        a plain streaming kernel that reads and writes B bytes

Kernel names are compared in the short form the library's profiler reports
(`conv3x3_direct<32, 1, 8, 16, 1, 4, 4, true>`): namespaces, a leading
`void` and the parameter list are dropped from the trace's names.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def short_name(name: str) -> str:
    s = name.replace("(anonymous namespace)::", "").replace("psw::", "").strip()
    if s.startswith("void "):
        s = s[5:]
    depth = 0
    for i, ch in enumerate(s):  # cut at the parameter list: the first '(' outside template brackets
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return s[:i].strip()
    return s


def kernel_stats(path: str):
    rows = []
    with open(path) as f:
        for r in csv.DictReader(f):
            rows.append({"name": short_name(r["Name"]), "calls": int(r["Calls"]),
                         "total_ns": float(r["TotalDurationNs"]), "avg_ns": float(r["AverageNs"]),
                         "min_ns": float(r["MinNs"]), "max_ns": float(r["MaxNs"])})
    rows.sort(key=lambda r: -r["total_ns"])
    return rows


def pmc_values(path: str, counter: str):
    """{short kernel name: [counter value per dispatch]} of a --pmc run."""
    out = defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            if r.get("Counter_Name") != counter:
                continue
            out[short_name(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return dict(out)


def kernel_sources(kernel: str):
    """Source files (relative to the repository) that define a library kernel."""
    base = "paper_1912_12675_amd/csrc/"
    if kernel.startswith(("conv3x3_direct", "conv3x3_dgrad_s2")):
        f = "direct.hip"
    elif kernel.startswith("conv3x3_wgrad"):
        f = "wgrad.hip"
    elif kernel.startswith(("igemm_kernel", "reduce_splits")):
        f = "conv.hip"
    else:
        f = "ops.hip"
    return [base + f, base + "internal.h"]


def source_hash(files) -> str:
    """sha256 over the given files (name and content, in the given order)."""
    h = hashlib.sha256()
    for f in files:
        h.update(f.encode())
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _mean(v):
    return sum(v) / len(v)


def traffic(kernels, fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, copy_kernel, copy_bytes):
    def pick(vals, sub):
        keys = [k for k in vals if sub in k]
        if len(keys) != 1:
            raise SystemExit(f"expected one kernel matching {sub!r}, found {keys}")
        return keys[0], vals[keys[0]]

    fk = pmc_values(fetch_csv, "FETCH_SIZE")
    wk = pmc_values(write_csv, "WRITE_SIZE")
    cname, cf = pick(pmc_values(copy_fetch_csv, "FETCH_SIZE"), copy_kernel)
    _, cw = pick(pmc_values(copy_write_csv, "WRITE_SIZE"), copy_kernel)
    # counters are in KiB per dispatch; scale each so the copy reads/writes copy_bytes
    f_scale = copy_bytes / (1024.0 * _mean(cf))
    w_scale = copy_bytes / (1024.0 * _mean(cw))
    out = {"copy_kernel": cname, "copy_bytes": copy_bytes, "copy_fetch_kib": _mean(cf), "copy_write_kib": _mean(cw),
           "fetch_scale": f_scale, "write_scale": w_scale, "kernels": {}}
    for kernel in kernels:
        if kernel not in fk or kernel not in wk:
            raise SystemExit(f"{kernel!r} not in the counter runs")
        fetch = 1024.0 * _mean(fk[kernel]) * f_scale
        write = 1024.0 * _mean(wk[kernel]) * w_scale
        out["kernels"][kernel] = {
            "bytes_per_launch": fetch + write, "fetch_bytes_per_launch": fetch, "write_bytes_per_launch": write,
            "fetch_kib_per_dispatch": _mean(fk[kernel]), "write_kib_per_dispatch": _mean(wk[kernel]),
            "dispatches": [len(fk[kernel]), len(wk[kernel])], "sources": kernel_sources(kernel),
            "source_sha256": source_hash(kernel_sources(kernel))}
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("csv")
    a.add_argument("--steps", type=int, required=True)
    a.add_argument("--top", type=int, default=25)
    b = sub.add_parser("traffic")
    b.add_argument("--kernel", action="append", required=True)
    for k in ("fetch", "write", "copy_fetch", "copy_write", "copy_kernel"):
        b.add_argument("--" + k.replace("_", "-"), required=True)
    b.add_argument("--copy-bytes", type=int, required=True)
    b.add_argument("--out")
    args = ap.parse_args(argv)
    if args.cmd == "stats":
        rows = kernel_stats(args.csv)
        tot = sum(r["total_ns"] for r in rows)
        print(f"| kernel | calls/step | mean us | us/step | share |\n|---|---:|---:|---:|---:|")
        for r in rows[:args.top]:
            print(f"| `{r['name']}` | {r['calls'] / args.steps:.2f} | {r['avg_ns'] / 1e3:.2f} | "
                  f"{r['total_ns'] / args.steps / 1e3:.1f} | {100 * r['total_ns'] / tot:.1f}% |")
        print(f"\nall kernels: {tot / args.steps / 1e6:.4f} ms/step over {args.steps} steps")
    else:
        t = traffic(args.kernel, args.fetch, args.write, args.copy_fetch, args.copy_write, args.copy_kernel,
                    args.copy_bytes)
        s = json.dumps(t, indent=1)
        if args.out:
            with open(args.out, "w") as f:
                f.write(s + "\n")
        print(s)


if __name__ == "__main__":
    sys.exit(main())
