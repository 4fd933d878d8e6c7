"""Summaries of rocprofv3 output for the kernels of libpsw.

    python -m paper_1912_12675_amd.rocprof_summary stats KERNEL_STATS_CSV --steps N [--top 25]
        per-kernel table (calls per step, mean / total time) of a
        `rocprofv3 --kernel-trace --stats --output-format csv` run

    python -m paper_1912_12675_amd.rocprof_summary replays KERNEL_TRACE_CSV --bench BENCH_JSON [--reps 20]
        the kernel-timing pass of bench.py in a `rocprofv3 --kernel-trace`
        run of the same command: runs of `reps` consecutive dispatches of one
        kernel on one queue are its isolated replays; per kernel, the trace's
        mean duration (end - start) and mean period (start to the next
        replay's start, i.e. duration + dispatch gap) beside bench.py's event
        time per launch for the same kernel

    python -m paper_1912_12675_amd.rocprof_summary mfma PMC_CSV --bench BENCH_JSON [--cycles 32] [--clock 2.4]
        matrix-core busy cycles per launch of every conv kernel from a
        `--pmc SQ_VALU_MFMA_BUSY_CYCLES ...` run, against the algorithmic
        instruction count (flop_per_launch / 2048 per 16x16x4 fp32 MFMA, times
        --cycles) and as a share of the SIMD-cycles of bench.py's launch time
        (busy / (avg_launch_us * clock * 1024 SIMDs))

    python -m paper_1912_12675_amd.rocprof_summary traffic --kernel NAME [--kernel NAME ...] \
            --fetch PMC_CSV --write PMC_CSV --copy-fetch PMC_CSV --copy-write PMC_CSV \
            --copy-kernel SUBSTRING --copy-bytes B --workload KEY [--out profiles/traffic.json]
        HBM bytes per launch of each kernel NAME from two `--pmc FETCH_SIZE`
        and `--pmc WRITE_SIZE` runs of one workload, each counter scaled by
        what it reads for a plain streaming kernel that reads and writes B
        bytes; --out keeps one section per workload KEY (bench.py's
        `traffic_key`: the same kernel moves other bytes at another batch)
        and replaces only this workload's

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


def replay_runs(trace_csv: str, reps: int):
    """{short kernel name: (durations_ns, periods_ns)} over the dispatches
    that belong to runs of at least `reps` consecutive dispatches of the same
    kernel on the same queue (the replays of bench.py's kernel-timing pass;
    no kernel of the training step repeats itself like that)."""
    by_queue = defaultdict(list)
    with open(trace_csv) as f:
        for r in csv.DictReader(f):
            by_queue[r["Queue_Id"]].append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]),
                                            short_name(r["Kernel_Name"])))
    out = defaultdict(lambda: ([], []))
    for q, ds in by_queue.items():
        ds.sort()
        i = 0
        while i < len(ds):
            j = i
            while j + 1 < len(ds) and ds[j + 1][2] == ds[i][2]:
                j += 1
            if j - i + 1 >= reps:
                dur, per = out[ds[i][2]]
                for k in range(i, j + 1):
                    dur.append(ds[k][1] - ds[k][0])
                    if k < j:
                        per.append(ds[k + 1][0] - ds[k][0])
            i = j + 1
    return dict(out)


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
    m = sub.add_parser("mfma")
    m.add_argument("csv")
    m.add_argument("--bench", required=True)
    m.add_argument("--cycles", type=int, default=32)
    m.add_argument("--clock", type=float, default=2.4, help="GHz")
    c = sub.add_parser("replays")
    c.add_argument("trace")
    c.add_argument("--bench", required=True, help="the JSON line bench.py printed in the same run")
    c.add_argument("--reps", type=int, default=20)
    b = sub.add_parser("traffic")
    b.add_argument("--kernel", action="append", required=True)
    for k in ("fetch", "write", "copy_fetch", "copy_write", "copy_kernel"):
        b.add_argument("--" + k.replace("_", "-"), required=True)
    b.add_argument("--copy-bytes", type=int, required=True)
    b.add_argument("--workload", required=True, help="section key, as bench.py's traffic_key")
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
    elif args.cmd == "mfma":
        with open(args.bench) as f:
            bench = json.loads([l for l in f if l.startswith("{")][-1])
        busy = pmc_values(args.csv, "SQ_VALU_MFMA_BUSY_CYCLES")
        print("| kernel | launches/step | MFMA busy cycles per launch | algorithmic instructions x cycles | "
              "launch us (bench) | busy share |\n|---|---:|---:|---:|---:|---:|")
        for k in bench["kernels"]:
            if not k["kind"].startswith("conv") or k["kernel"] not in busy:
                continue
            b = _mean(busy[k["kernel"]])
            alg = k["flop_per_launch"] / 2048.0 * args.cycles
            share = b / (k["avg_launch_us"] * 1e-6 * args.clock * 1e9 * 1024)
            print(f"| `{k['kernel']}` | {k['launches_per_step']:.2f} | {b:,.0f} | {alg:,.0f} | {k['avg_launch_us']:.2f} | "
                  f"{100 * share:.1f}% |")
    elif args.cmd == "replays":
        with open(args.bench) as f:
            line = [l for l in f if l.startswith("{")][-1]
        bench = json.loads(line)
        every = {k["kernel"]: k for k in bench.get("kernels", [])}
        ev = {k: v["avg_launch_us"] for k, v in every.items()}
        roof = bench.get("roofline") or {}
        runs = replay_runs(args.trace, args.reps)
        print("| kernel | replays | trace mean duration us | trace mean period us | bench events us/launch | "
              "events / period | events / duration |\n|---|---:|---:|---:|---:|---:|---:|")
        for name in sorted(runs, key=lambda n: -_mean(runs[n][0]) * len(runs[n][0])):
            dur, per = runs[name]
            d, p_ = _mean(dur) / 1e3, (_mean(per) / 1e3 if per else float("nan"))
            e = ev.get(name)
            es = f"{e:.2f} | {e / p_:.3f} | {e / d:.3f}" if e else "- | - | -"
            print(f"| `{name}` | {len(dur)} | {d:.2f} | {p_:.2f} | {es} |")
        # the conv matrix-core figure and the dominant kernel's roofline, from
        # the trace's durations and from bench's event times
        conv = [k for k in every.values() if k["kind"] in ("conv_fwd", "conv_bwd_data", "conv_bwd_weight")]
        if conv and all(k["kernel"] in runs for k in conv):
            flop = sum(k["launches_per_step"] * k["flop_per_launch"] for k in conv)
            t_tr = sum(k["launches_per_step"] * _mean(runs[k["kernel"]][0]) * 1e-9 for k in conv)
            t_ev = sum(k["launches_per_step"] * k["avg_launch_us"] * 1e-6 for k in conv)
            peak = (bench.get("conv_mfma") or {}).get("peak", 157.3)
            print(f"\nconv kernels per step: {flop / 1e9:.3f} GFLOP; summed time {t_tr * 1e6:.1f} us (trace "
                  f"durations) / {t_ev * 1e6:.1f} us (bench events): {flop / t_tr / 1e12:.2f} / "
                  f"{flop / t_ev / 1e12:.2f} TFLOP/s = {flop / t_tr / 1e12 / peak:.4f} / "
                  f"{flop / t_ev / 1e12 / peak:.4f} of {peak} TFLOP/s")
        if roof.get("kernel") in runs and roof["kernel"] in every:
            k = every[roof["kernel"]]
            d = _mean(runs[roof["kernel"]][0]) * 1e-9
            work = k["flop_per_launch"] if roof["bound"] == "mfma" else k["bytes_per_launch"]
            scale = 1e12 if roof["bound"] == "mfma" else 1e9
            print(f"dominant kernel `{roof['kernel']}` ({roof['bound']}): {work / d / scale:.1f} {roof['unit']} "
                  f"from the trace's mean duration {d * 1e6:.2f} us = {work / d / scale / roof['peak']:.4f} of peak; "
                  f"bench: {roof['achieved']} {roof['unit']} = {roof['frac']}")
    else:
        t = traffic(args.kernel, args.fetch, args.write, args.copy_fetch, args.copy_write, args.copy_kernel,
                    args.copy_bytes)
        base = {"workloads": {}}
        if args.out and os.path.exists(args.out):
            with open(args.out) as f:
                base = json.load(f)
        base.setdefault("workloads", {})[args.workload] = t
        s = json.dumps(base, indent=1)
        if args.out:
            with open(args.out, "w") as f:
                f.write(s + "\n")
        print(s)


if __name__ == "__main__":
    sys.exit(main())
