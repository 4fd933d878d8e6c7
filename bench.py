"""Benchmark: stale-weight pipelined training of ResNet-20 (CIFAR shape,
batch 128) on one MI355X through libpsw.

One step = one mini-batch through all 4 stages: forward (PPV (7,13,19),
weights of version t - d_s with d = [3,2,1,0]), softmax cross-entropy,
backward (weight gradients + data gradients with the current weights), and
the SGD-momentum update into each stage's weight-version ring.  The steps
run as the paper's pipeline on one GPU: the forward pass of mini-batch t+1
overlaps the backward pass of mini-batch t where the stale weights allow it
(psw_pipeline_run; results identical to one psw_stage_step call per step).
By default the timed steps are one eager psw_pipeline_run call; --mode
graph replays a HIP graph that captured one period (lcm of the ring depths
and of the 3 step sets = 12 steps) of the pipeline, --mode sequential makes one
psw_stage_step call per step; the modes not selected are timed over K more
steps for context (on ROCm 7.2 the graph replays of this three-stream
pipeline run slower than issuing it eagerly).  Inputs
are synthetic N(0,1) [128,3,32,32] batches with uniform labels, all resident
in HBM before timing starts.

Prints one JSON line.  `value` is images/s over the K timed steps.
`memory` is the device memory the net holds; `--step-sets 2` runs the
pipeline with one step set less (the forward pass of step t then waits for
the weight stream's step t-2 instead of t-3).
`--bf16` runs the same ResNet-20 configuration with bf16 products (fp32
accumulation); `--workload resnet110` runs ResNet-110 at batch 256 with bf16
products, 8 stages of [7,7,7,7,7,7,6,6] blocks and staleness d_s = 7 - s
(50 timed steps by default; its ring period of 840 steps is not captured
as a graph).  Both report the conv kernels against HBM beside bf16 MFMA.

Measurement, in order: W warm-up steps (eager, including the pipeline
fill), the graph capture and one untimed replay; the K timed steps (wall
clock, no events); the other modes; then a kernel-timing pass of
REPLAY_STEPS eager pipelined steps of the same workload in which every
kernel launch is replayed in isolation (psw_net_profile_replay): the
library waits for the device to be idle, then issues the launch REPLAY_REPS
times back to back on its stream between one start / stop event pair.  The
mean per launch is the kernel's own duration plus the dispatch gap between
consecutive launches of one stream, with no event-pair cost in it and no
other stream's kernels beside it; a rocprofv3 kernel trace of the same
command shows each replay as its own dispatch (paper_1912_12675_amd/
rocprof_summary.py --replays pairs them up).  That pass gives the per-kernel
table, the conv matrix-core figure the metric names (algorithmic conv FLOPs
per step / summed conv kernel time per step) and the dominant kernel
(largest summed time per step): `roofline.achieved` = its algorithmic work
per launch / its mean launch time.  `conv_mfma.in_step` is the conv FLOPs
per step over the whole step time instead (all kernels of the three
streams sharing the chip).  `roofline.traffic` is the HBM bytes per launch
from rocprofv3 FETCH_SIZE / WRITE_SIZE counters (calibrated on a plain
streaming kernel) stored in profiles/traffic.json under the workload's
key (`traffic_key`), used only when the source files defining that kernel
still hash to what was profiled, else null.
`cpu_baseline` times the CPU oracle on a bounded sample: 2-step runs of the
same workload, repeated until 10 s of host time have passed (about 12 steps
on 16 host threads).

`python bench.py --copy-calibration` instead runs a plain streaming kernel
five times: y = -x over 256 MiB (reads and writes 256 MiB each; the
reference kernel for the counter scale).
"""
from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "training images/sec at 1 GPU (ResNet-20, batch 128) + conv MFMA % of peak"
METRIC_R110 = "training images/sec at 1 GPU (ResNet-110, batch 256, bf16 products) + conv MFMA % of peak"
PEAK_FP32_MFMA = 157.3   # TFLOP/s, MI355X dense fp32 matrix
PEAK_BF16_MFMA = 2500.0  # TFLOP/s, MI355X dense bf16 matrix
PEAK_HBM = 8000.0        # GB/s, MI355X HBM3E
REPLAY_STEPS = 3   # pipelined steps of the kernel-timing pass
REPLAY_REPS = 20   # back-to-back launches per recorded launch
COPY_BYTES = 256 << 20


def traffic_key(wl):
    """Section of profiles/traffic.json for a workload: one kernel moves other
    bytes at another batch size (resnet20_b128, resnet20_bf16_b128,
    resnet110_bf16_b256)."""
    return f"{wl.name}_b{wl.batch}"


def measured_traffic(kernel, key):
    """HBM bytes per launch of `kernel` in workload section `key` of
    profiles/traffic.json, or None when the file has no entry for it or the
    entry was taken on other sources of that kernel (each entry records which
    source files define the kernel and their hash)."""
    import hashlib

    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    t = t.get("workloads", {}).get(key, {}).get("kernels", {}).get(kernel)
    if not t or not t.get("sources"):
        return None
    h = hashlib.sha256()
    for rel in t["sources"]:
        h.update(rel.encode())
        try:
            with open(os.path.join(ROOT, rel), "rb") as fh:
                h.update(fh.read())
        except OSError:
            return None
    if h.hexdigest() != t.get("source_sha256"):
        return None
    return t.get("bytes_per_launch")


def roofline_of(k, peak_flops):
    """Roofline entry of one kernel's profile record (summed over launches)."""
    t_s = k["ms"] * 1e-3
    # the binding roof: the one the algorithmic work needs longer at
    mfma = k["flops"] / (peak_flops * 1e12) >= k["bytes"] / (PEAK_HBM * 1e9)
    if mfma:
        ach = k["flops"] / t_s / 1e12
        return {"bound": "mfma", "achieved": round(ach, 3), "peak": peak_flops, "unit": "TFLOP/s",
                "frac": round(ach / peak_flops, 4)}
    ach = k["bytes"] / t_s / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM, "unit": "GB/s",
            "frac": round(ach / PEAK_HBM, 4)}


def copy_calibration():
    import torch

    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "launches": 5}), flush=True)


def host_cpu():
    """Model name of the host CPU and the number of logical CPUs this process may use."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"model": model, "logical_cpus_available": len(os.sched_getaffinity(0))}


def cpu_baseline(wl, chunk=2, min_seconds=10.0, max_chunks=15):
    from oracle import oracle
    from paper_1912_12675_amd import synth

    oracle.build()
    p0 = synth.init_params(wl)
    xs, ys = synth.batches(wl, chunk)
    steps, t0 = 0, time.perf_counter()
    while steps < chunk * max_chunks:
        oracle.train(wl.ops, wl.in_shape, wl.stage_end, p0, xs, ys, wl.staleness(chunk), wl.lr_table(chunk),
                     wl.momentum, wl.weight_decay, wl.nesterov, bf16=wl.bf16)
        steps += chunk
        if time.perf_counter() - t0 >= min_seconds:
            break
    dt = time.perf_counter() - t0
    cores = oracle.num_threads()
    # one step on one host thread, for the single-threaded figure
    oracle.set_threads(1)
    try:
        t1 = time.perf_counter()
        oracle.train(wl.ops, wl.in_shape, wl.stage_end, p0, xs[:1], ys[:1], wl.staleness(1), wl.lr_table(1),
                     wl.momentum, wl.weight_decay, wl.nesterov, bf16=wl.bf16)
        dt1 = time.perf_counter() - t1
    finally:
        oracle.set_threads(cores)
    return {"value": round(steps * wl.batch / dt, 3), "unit": "images/s", "cores": cores,
            "kind": "oracle", "host": host_cpu(),
            "sample": f"{steps} stale-weight training steps of the same workload ({wl.name}, batch {wl.batch}, "
                      f"float64 direct loops, OpenMP; runs of {chunk} steps until {min_seconds:.0f} s or "
                      f"{chunk * max_chunks} steps), {dt:.1f} s",
            "single_thread": {"value": round(wl.batch / dt1, 3), "unit": "images/s", "cores": 1,
                              "sample": f"1 step of the same workload on one thread, {dt1:.1f} s"}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default 100; resnet110: 50)")
    ap.add_argument("--warmup", type=int, default=None, help="warm-up steps (default 20; resnet110: 10)")
    ap.add_argument("--workload", choices=("resnet20", "resnet110"), default="resnet20",
                    help="resnet20: ResNet-20, batch 128, 4 stages, d = [3,2,1,0] (the metric's configuration); "
                         "resnet110: ResNet-110, batch 256, bf16 products, 8 stages, d_s = 7 - s")
    ap.add_argument("--bf16", action="store_true", help="bf16-in / fp32-accumulate conv and FC products")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--mode", choices=("pipelined", "graph", "sequential"), default="pipelined",
                    help="pipelined: psw_pipeline_run issued eagerly (default); graph: the same steps replayed "
                         "from a captured HIP graph; sequential: one psw_stage_step call per step")
    ap.add_argument("--step-sets", type=int, choices=(2, 3), default=3,
                    help="step sets the pipelined run rotates: 3 (default) lets the forward pass of step t wait "
                         "for the weight stream's step t-3, 2 for its step t-2, at one step set less memory")
    ap.add_argument("--no-profile", action="store_true",
                    help="no events at all: skip the kernel-timing pass")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a plain 256 MiB streaming kernel 5 times (counter calibration) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the library has no multi-GPU path; "
              "the pipeline's stages all run on a single MI355X.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1912_12675_amd import psw, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        copy_calibration()
        return
    r110 = args.workload == "resnet110"
    wl = synth.resnet110_workload() if r110 else synth.resnet20_workload(bf16=args.bf16)
    K = args.steps if args.steps is not None else (50 if r110 else 100)
    W = args.warmup if args.warmup is not None else (10 if r110 else 20)
    period = args.step_sets  # step sets of the pipelined run
    for d in wl.ring_depth():
        period = period * d // math.gcd(period, d)
    # a graph replays one period of ring slots and step sets: 12 steps for
    # ResNet-20's rings [4,3,2,1], 840 for ResNet-110's [8..1] (not captured)
    use_graph = period <= 64
    if not use_graph and args.mode == "graph":
        print(f"--mode graph: the pipeline's period is {period} steps, too long to capture", file=sys.stderr)
        sys.exit(2)
    T = W + period + REPLAY_STEPS + 3 * K + period
    net = psw.Net(wl.ops, wl.batch, wl.in_shape, wl.stage_end, wl.ring_depth(T), bf16=wl.bf16,
                  step_sets=args.step_sets)
    net.load_params(synth.init_params(wl))
    stal = wl.staleness(T)
    # every mini-batch resident in HBM before timing (a fresh batch per step)
    n_distinct = min(T, 64)
    xs = torch.empty((n_distinct, wl.batch) + tuple(wl.in_shape), dtype=torch.float32, device="cuda")
    ys = torch.empty((n_distinct, wl.batch), dtype=torch.int32, device="cuda")
    for i in range(n_distinct):
        x, y = synth.batch(wl, i)
        xs[i].copy_(torch.from_numpy(x))
        ys[i].copy_(torch.from_numpy(y))
    torch.cuda.synchronize()
    t = 0
    losses = torch.zeros(max(K, W, REPLAY_STEPS, 1), dtype=torch.float32, device="cuda")
    nb = ctypes.c_int64()
    psw._check(psw.lib().psw_net_pipeline_bytes(net.handle, ctypes.byref(nb)))
    net_step_bytes = nb.value

    def run_sequential(n):
        nonlocal t
        for _ in range(n):
            net.step(t, stal[t], wl.lr, xs[t % n_distinct], ys[t % n_distinct], wl.momentum, wl.weight_decay,
                     wl.nesterov)
            t += 1

    def run_pipelined(n):
        # one call: step t+i uses batch i mod n_distinct
        nonlocal t
        net.pipeline_run(t, stal[t:t + n], wl.lr, xs, ys, losses[:n], wl.momentum, wl.weight_decay, wl.nesterov)
        t += n

    graph = None
    glosses = torch.zeros(period, dtype=torch.float32, device="cuda")

    gt0 = W  # the graph is captured at step W

    def run_graph(n):
        # eager steps until t is congruent to the capture step modulo the
        # period, replays of the captured period, the remainder eagerly
        nonlocal t
        align = min((gt0 - t) % period, n)
        if align:
            run_pipelined(align)
            n -= align
        for _ in range(n // period):
            graph.launch()
            t += period
        if n % period:
            run_pipelined(n % period)

    modes = {"graph": run_graph, "pipelined": run_pipelined, "sequential": run_sequential}
    if not use_graph:
        del modes["graph"]
    run = modes[args.mode]

    run_pipelined(W)  # includes the pipeline fill (versions clamped at 0)
    if use_graph:
        graph = net.capture(stal[t:t + period], wl.lr, xs, ys, glosses, wl.momentum, wl.weight_decay, wl.nesterov)
        run_graph(period)  # first replay uploads the graph
    torch.cuda.synchronize()
    # timed region: no events
    t0 = time.perf_counter()
    run(K)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    if args.mode == "sequential":
        loss = float(net.loss.item())
    elif args.mode == "graph" and K % period == 0:
        loss = float(glosses[-1].item())
    else:  # the last call was an eager pipelined run of K (or K mod period) steps
        loss = float(losses[(K if args.mode == "pipelined" else K % period) - 1].item())
    assert np.isfinite(loss), loss
    ms_per_step = 1000.0 * elapsed / K
    img_s = wl.batch * K / elapsed
    # the other execution modes, for context (same workload, continuing the run)
    others = {}
    for name, fn in modes.items():
        if name == args.mode:
            continue
        t1 = time.perf_counter()
        fn(K)
        torch.cuda.synchronize()
        others[name] = round(wl.batch * K / (time.perf_counter() - t1), 2)

    # kernel-timing pass over the same workload (eager pipelined: graphs carry
    # no events): every launch replayed REPLAY_REPS times in isolation
    peak = PEAK_BF16_MFMA if wl.bf16 else PEAK_FP32_MFMA
    kernels, breakdown, conv, roof = [], None, None, None
    KP = REPLAY_STEPS if not args.no_profile else 0
    if KP:
        net.profile(True)
        net.profile_replay(REPLAY_REPS)
        run_pipelined(KP)
        torch.cuda.synchronize()
        kernels = sorted(net.profile_kernels(), key=lambda k: -k["ms"])
        net.profile_replay(1)
        net.profile(False)
        kinds = {}
        for k in kernels:
            kinds[k["kind"]] = kinds.get(k["kind"], 0.0) + k["ms"]
        breakdown = {k: round(v / KP, 4) for k, v in kinds.items()}
        ck = [k for k in kernels if k["kind"] in ("conv_fwd", "conv_bwd_data", "conv_bwd_weight")]
        conv_ms = sum(k["ms"] for k in ck) / KP
        conv_flop = sum(k["flops"] for k in ck) / KP
        ach = conv_flop / (conv_ms * 1e-3) / 1e12
        in_step = conv_flop / (ms_per_step * 1e-3) / 1e12
        conv = {"achieved": round(ach, 3), "peak": peak, "unit": "TFLOP/s", "frac": round(ach / peak, 4),
                "flop_per_step": conv_flop, "conv_kernel_ms_per_step": round(conv_ms, 4),
                "conv_kernel_launches_per_step": sum(k["launches"] for k in ck) / KP,
                "in_step": {"achieved": round(in_step, 3), "frac": round(in_step / peak, 4),
                            "what": "conv FLOPs per step / ms_per_step of the timed run"},
                "what": "all convolution kernels (forward, backward-data with fused BN sums or folded BN backward, "
                        "backward-weight): algorithmic conv FLOPs / summed kernel time, each kernel timed in "
                        f"isolation as {REPLAY_REPS} back-to-back launches; the backward-weight split partial sums "
                        "are reduced inside the stage update kernel (sgd_stage_k), counted in frac_with_update"}
        uk = [k for k in kernels if k["name"] == "sgd_stage_k"]
        if uk:
            ums = conv_ms + sum(k["ms"] for k in uk) / KP
            conv["frac_with_update"] = round(conv_flop / (ums * 1e-3) / 1e12 / peak, 4)
        # the same kernels against HBM: their algorithmic bytes over their time
        # (the binding roof of the bf16 mode, whose tensors stay fp32 in HBM)
        conv_bytes = sum(k["bytes"] for k in ck) / KP
        gbs = conv_bytes / (conv_ms * 1e-3) / 1e9
        conv["hbm"] = {"achieved": round(gbs, 1), "peak": PEAK_HBM, "unit": "GB/s", "frac": round(gbs / PEAK_HBM, 4),
                       "bytes_per_step": conv_bytes}
        d = kernels[0]  # the dominant kernel: largest summed time
        roof = roofline_of(d, peak)
        roof["traffic"] = measured_traffic(d["name"], traffic_key(wl))
        roof.update({"kernel": d["name"], "launches": d["launches"],
                     "avg_launch_us": round(1e3 * d["ms"] / d["launches"], 3),
                     "flop_per_launch": d["flops"] / d["launches"], "bytes_per_launch": d["bytes"] / d["launches"],
                     "timed_over": f"{KP} pipelined steps of the same workload after the timed region; every launch "
                                   f"replayed {REPLAY_REPS} times back to back on its stream with the device "
                                   "otherwise idle, between one start/stop HIP event pair; avg_launch_us = the "
                                   f"pair's time / {REPLAY_REPS}"})
    top = []
    for k in kernels[:10]:
        r = roofline_of(k, peak)
        top.append({"kernel": k["name"], "kind": k["kind"], "launches_per_step": k["launches"] / KP,
                    "us_per_step": round(1e3 * k["ms"] / KP, 2), "avg_launch_us": round(1e3 * k["ms"] / k["launches"], 3),
                    "bound": r["bound"], "achieved": r["achieved"], "unit": r["unit"], "frac": r["frac"],
                    "bytes_per_launch": k["bytes"] / k["launches"], "traffic": measured_traffic(k["name"], traffic_key(wl))})

    every = [{"kernel": k["name"], "kind": k["kind"], "launches_per_step": k["launches"] / KP,
              "avg_launch_us": round(1e3 * k["ms"] / k["launches"], 3), "flop_per_launch": k["flops"] / k["launches"],
              "bytes_per_launch": k["bytes"] / k["launches"]} for k in kernels]
    out = {
        "metric": METRIC_R110 if r110 else METRIC,
        "value": round(img_s, 2),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16-in/f32-acc" if wl.bf16 else "f32",
        "data": "synthetic",
        "config": {"workload": ("ResNet-110 (CIFAR shape), batch 256, bf16 products with fp32 accumulation, 8 stages "
                                "of [7,7,7,7,7,7,6,6] blocks, staleness d_s = 7 - s, SGD momentum 0.9, lr 0.01" if r110
                                else "ResNet-20 (CIFAR shape), batch 128, 4 stages at PPV (7,13,19), staleness "
                                     "[3,2,1,0], SGD momentum 0.9, lr 0.01"),
                   "global_batch": wl.batch, "input": "3x32x32 N(0,1)", "parallelism": "single GPU, all stages",
                   "execution": {"graph": f"pipelined (forward of t+1 overlaps backward of t), replayed from a "
                                          f"HIP graph of {period} captured steps",
                                 "pipelined": "pipelined psw_pipeline_run issued eagerly",
                                 "sequential": "one psw_stage_step call per step"}[args.mode]},
        "other_modes_images_per_s": others,
        "memory": {"step_sets": args.step_sets, "step_set_bytes": net_step_bytes, "arena_bytes": net.arena_bytes,
                   "ring_bytes": 4 * net.ring_floats, "device_bytes": net.device_bytes(),
                   "what": "device memory of the net: weight-version rings, momentum, gradients, running "
                           "statistics, the arena (one step set: activations, saved statistics, every tensor's "
                           "gradient; and the shared workspaces) and the pipelined run's extra step sets"},
        "roofline": roof,
        "conv_mfma": conv,
        "kernel_ms_per_step": breakdown,
        "top_kernels": top,
        "kernels": every,
        "final_loss": round(loss, 5),
    }
    if not args.no_cpu_baseline:
        # the same workload; ResNet-110's steps take ~20 s of oracle time each
        out["cpu_baseline"] = cpu_baseline(wl, chunk=1, max_chunks=1) if r110 else cpu_baseline(wl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
