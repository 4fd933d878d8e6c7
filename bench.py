"""Benchmark: stale-weight pipelined training of ResNet-20 (CIFAR shape,
batch 128) on one MI355X through libpsw.

One step = psw_stage_step on one mini-batch: forward of all 4 stages (PPV
(7,13,19), weights of version t - d_s with d = [3,2,1,0]), softmax
cross-entropy, backward (weight gradients + data gradients with the current
weights), and the SGD-momentum update into each stage's weight-version ring.
Inputs are synthetic N(0,1) [128,3,32,32] batches with uniform labels, all
resident in HBM before timing starts.

Prints one JSON line.  `value` is images/s over the K timed steps.
`roofline` reports the convolution kernels (forward, backward-data,
backward-weight: the matrix-core work of the path) against the fp32 MFMA
peak, timed with HIP events recorded on the step's stream around every conv
launcher during a second run of K steps.  `cpu_baseline` times the CPU oracle
on a bounded sample (2 steps of the same workload).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "training images/sec at 1 GPU (ResNet-20, batch 128) + conv MFMA % of peak"
PEAK_FP32_MFMA = 157.3   # TFLOP/s, MI355X dense fp32 matrix
PEAK_BF16_MFMA = 2500.0  # TFLOP/s, MI355X dense bf16 matrix


def shapes(ops, batch, in_shape):
    """Output shape of every tensor (tensor 0 = the batch)."""
    t = [(batch,) + tuple(in_shape)]
    for o in ops:
        kind, in0, _, cin, cout, k, st, pad, _ = (int(v) for v in o)
        n, c, h, w = t[in0]
        if kind == 1:
            t.append((n, cout, (h + 2 * pad - k) // st + 1, (w + 2 * pad - k) // st + 1))
        elif kind == 2:
            t.append((n, c, h, w))
        elif kind == 3:
            t.append((n, c, (h - k) // st + 1, (w - k) // st + 1))
        elif kind == 4:
            t.append((n, c, 1, 1))
        else:
            t.append((n, cout, 1, 1))
    return t


def conv_flops(ops, batch, in_shape):
    """Algorithmic FLOPs of the conv passes of one step: 2*N*K*P*Q*C*R*S for
    the forward, the backward-weight, and the backward-data pass (none for a
    conv that reads the input batch)."""
    t = shapes(ops, batch, in_shape)
    fwd = bwd_w = bwd_d = 0
    for i, o in enumerate(ops):
        kind, in0, _, cin, cout, k, _, _, _ = (int(v) for v in o)
        if kind != 1:
            continue
        n, kk, p, q = t[i + 1]
        f = 2 * n * kk * p * q * cin * k * k
        fwd += f
        bwd_w += f
        if in0 > 0:
            bwd_d += f
    return fwd, bwd_d, bwd_w


def cpu_baseline(wl, steps=2):
    from oracle import oracle
    from paper_1912_12675_amd import synth

    oracle.build()
    p0 = synth.init_params(wl)
    xs, ys = synth.batches(wl, steps)
    t0 = time.perf_counter()
    oracle.train(wl.ops, wl.in_shape, wl.stage_end, p0, xs, ys, wl.staleness(steps), wl.lr, wl.momentum,
                 wl.weight_decay, wl.nesterov, bf16=wl.bf16)
    dt = time.perf_counter() - t0
    return {"value": round(steps * wl.batch / dt, 3), "unit": "images/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{steps} stale-weight training steps of the same workload (ResNet-20, batch {wl.batch}, "
                      f"float64 direct loops, OpenMP), {dt:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--bf16", action="store_true", help="bf16-in / fp32-accumulate conv and FC products")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip the event-timed second pass")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): this build has no multi-GPU path; "
              "the pipeline's stages all run on a single MI355X.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1912_12675_amd import psw, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    wl = synth.resnet20_workload(bf16=args.bf16)
    K, W = args.steps, args.warmup
    T = K * (1 if args.no_profile else 2) + W
    net = psw.Net(wl.ops, wl.batch, wl.in_shape, wl.stage_end, wl.ring_depth(T), bf16=wl.bf16)
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

    def run(n):
        nonlocal t
        for _ in range(n):
            net.step(t, stal[t], wl.lr, xs[t % n_distinct], ys[t % n_distinct], wl.momentum, wl.weight_decay,
                     wl.nesterov)
            t += 1

    run(W)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(K)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    loss = float(net.loss.item())
    assert np.isfinite(loss), loss
    ms_per_step = 1000.0 * elapsed / K
    img_s = wl.batch * K / elapsed

    fwd, bwd_d, bwd_w = conv_flops(wl.ops, wl.batch, wl.in_shape)
    conv_flop = fwd + bwd_d + bwd_w
    roof = None
    breakdown = None
    if not args.no_profile:
        net.profile(True)
        run(K)
        torch.cuda.synchronize()
        prof = net.profile_read()
        net.profile(False)
        breakdown = {k: round(v[0] / K, 4) for k, v in prof.items() if v[1]}
        conv_ms = sum(prof[k][0] for k in ("conv_fwd", "conv_bwd_data", "conv_bwd_weight")) / K
        launches = sum(prof[k][1] for k in ("conv_fwd", "conv_bwd_data", "conv_bwd_weight")) / K
        achieved = conv_flop / (conv_ms * 1e-3) / 1e12
        peak = PEAK_BF16_MFMA if wl.bf16 else PEAK_FP32_MFMA
        roof = {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": None,
                "kernel": "conv implicit-GEMM launchers (forward, backward-data, backward-weight), all layers",
                "flop_per_step": conv_flop, "conv_ms_per_step": round(conv_ms, 4),
                "conv_launches_per_step": launches}

    out = {
        "metric": METRIC,
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
        "config": {"workload": "ResNet-20 (CIFAR shape), batch 128, 4 stages at PPV (7,13,19), staleness [3,2,1,0], "
                               "SGD momentum 0.9, lr 0.01",
                   "global_batch": wl.batch, "input": "3x32x32 N(0,1)", "parallelism": "single GPU, all stages"},
        "roofline": roof,
        "kernel_ms_per_step": breakdown,
        "final_loss": round(loss, 5),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(synth.resnet20_workload(bf16=args.bf16))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
