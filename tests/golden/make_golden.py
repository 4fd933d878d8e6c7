"""Write the oracle's results for the full-size runs to tests/golden/.
Calls only the oracle and the seeded input generator; never the GPU path.

    python tests/golden/make_golden.py [fp32|bf16|alexnet|vgg16|resnet110|states_fp32|states_bf16 ...]

fp32 / bf16: ResNet-20, batch 128, 4 stages at the Table 1 PPV (7,13,19),
staleness [3,2,1,0], 50 steps, lr 0.01, momentum 0.9.  Stored: the
parameter update W^(50) - W^(0) (float32; W^(0) is regenerated from the
seed), the 50 losses and the version table.

states_fp32 / states_bf16: the same ResNet-20 run's state at steps 25 and
49 -- for every stage s the versions W_s^(t-d_s) .. W_s^(t) its ring holds
(d = [3,2,1,0]), the momentum and the BN running statistics, all rounded to
float32 -- so that a test can start one step from a point on the oracle's
own trajectory (the oracle run to 25, then resumed from its exact float64
state to 49).

alexnet / vgg16 / resnet110: the other full-size configurations (AlexNet-style
net, batch 128, 20 steps, split after conv2, staleness [2,0], App. A's rate
0.001 with Nesterov momentum and weight decay 0.004; VGG-16-BN,
batch 128, 30 stale steps at PPV (2,4,7) then 10 non-pipelined; ResNet-110,
batch 256, bf16 products, 8 stages with d_s = 7-s, the first 3 steps).
These nets have up to 86M parameters, so what is stored is: the losses, the
version table, the L2 norm of every parameter tensor and of its update, and
the values of a seeded sample of 200,000 final parameters.  Each is run twice:
on the inputs, and on the inputs moved one float32 ulp (seeded signs); the
distance between the two runs (the oracle's own sensitivity to rounding-level
changes, "spread") is stored beside the result and sets the test's bar where
it exceeds the target tolerance.
"""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from paper_1912_12675_amd import synth  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
SAMPLE = 200_000


def make(mode):
    wl = synth.resnet20_workload(bf16=(mode == "bf16"))
    T = wl.steps
    p0 = synth.init_params(wl)
    xs, ys = synth.batches(wl, T)
    t0 = time.time()
    out = O.train(wl.ops, wl.in_shape, wl.stage_end, p0, xs, ys, wl.staleness(T), wl.lr_table(T), wl.momentum,
                  wl.weight_decay, wl.nesterov, bf16=wl.bf16, dropout_seed=wl.dropout_seed)
    path = os.path.join(HERE, f"resnet20_b128_50steps_{mode}.npz")
    np.savez_compressed(path, delta=(out["params"] - p0.astype(np.float64)).astype(np.float32),
                        losses=out["losses"], versions=out["versions"])
    print(f"{mode}: {time.time() - t0:.0f} s, final loss {out['losses'][-1]:.6f} -> {path}", flush=True)


def sample_index(n):
    """Seeded, sorted sample of parameter indices (all of them when n <= SAMPLE)."""
    if n <= SAMPLE:
        return np.arange(n, dtype=np.int64)
    return np.sort(np.random.Generator(np.random.PCG64(20260)).choice(n, size=SAMPLE, replace=False))


def tensor_norms(wl, flat, p0):
    """Per parameter tensor: L2 norm of the final values, of the update, and
    whether the initial value is non-zero (zero-initialised tensors -- BN
    beta, biases -- hold only their update, so their norm is compared through
    the parameter sample instead)."""
    layout, counts = synth.param_layout(wl)
    base = np.concatenate([[0], np.cumsum(counts)])
    norms, dnorms, nz = [], [], []
    for op, name, shape, s, off in layout:
        i0 = int(base[s]) + off
        seg0 = p0[i0:i0 + int(np.prod(shape))]
        seg = flat[i0:i0 + int(np.prod(shape))]
        norms.append(np.linalg.norm(seg))
        dnorms.append(np.linalg.norm(seg - seg0))
        nz.append(np.linalg.norm(seg0) > 0.0)
    return np.array(norms), np.array(dnorms), np.array(nz)


def ulp_move(x, seed):
    """x moved one float32 ulp up or down elementwise (seeded signs)."""
    up = np.random.Generator(np.random.PCG64(seed)).random(x.shape) < 0.5
    return np.where(up, np.nextafter(x, np.float32(np.inf)), np.nextafter(x, np.float32(-np.inf))).astype(np.float32)


FULL = {
    "alexnet": (lambda: synth.alexnet_workload(), 20),
    "vgg16": (lambda: synth.vgg16_workload(), 40),
    "resnet110": (lambda: synth.resnet110_workload(), 3),
}


def make_full(name):
    factory, T = FULL[name]
    wl = factory()
    p0 = synth.init_params(wl).astype(np.float64)
    xs, ys = synth.batches(wl, T)
    st = wl.staleness(T)
    idx = sample_index(p0.size)
    res = []
    t0 = time.time()
    for x in (xs, ulp_move(xs, 1912)):
        out = O.train(wl.ops, wl.in_shape, wl.stage_end, p0, x, ys, st, wl.lr_table(T), wl.momentum,
                      wl.weight_decay, wl.nesterov, bf16=wl.bf16, dropout_seed=wl.dropout_seed)
        norms, dnorms, nz = tensor_norms(wl, out["params"], p0)
        res.append(dict(sample=out["params"][idx], norms=norms, dnorms=dnorms, nz=nz, losses=out["losses"],
                        versions=out["versions"]))
        print(f"{name}: run {len(res)} {time.time() - t0:.0f} s, final loss {out['losses'][-1]:.6f}", flush=True)
        del out
    a, b = res
    s0 = p0[idx]
    spread = dict(
        sample=np.linalg.norm(a["sample"] - b["sample"]) / np.linalg.norm(a["sample"]),
        update=np.linalg.norm(a["sample"] - b["sample"]) / max(np.linalg.norm(a["sample"] - s0), 1e-30),
        loss=np.abs(a["losses"] - b["losses"]).max() / np.abs(a["losses"]).max(),
        norm=np.max((np.abs(a["norms"] - b["norms"]) / np.maximum(a["norms"], 1e-30))[a["nz"]]))
    path = os.path.join(HERE, f"{name}_full_{T}steps.npz")
    np.savez_compressed(path, index=idx, sample=a["sample"], norms=a["norms"], dnorms=a["dnorms"], nonzero_init=a["nz"],
                        losses=a["losses"], versions=a["versions"], steps=T,
                        **{"spread_" + k: v for k, v in spread.items()})
    print(f"{name}: spread {spread} -> {path}", flush=True)


STATE_STEPS = (25, 49)


def make_states(mode):
    wl = synth.resnet20_workload(bf16=(mode == "bf16"))
    T = STATE_STEPS[-1]
    D = max(wl.ring_depth(T))
    p0 = synth.init_params(wl).astype(np.float64)
    xs, ys = synth.batches(wl, T)
    st, lr = wl.staleness(T), wl.lr_table(T)
    counts = O.param_counts(wl.ops, wl.in_shape, 1, wl.stage_end)
    depth = wl.ring_depth(T)
    out, t_prev, res = {}, 0, None
    t0 = time.time()
    for t in STATE_STEPS:
        if res is None:
            hist0, mom0, rm, rv = [[v] for v in np.split(p0, np.cumsum(counts)[:-1])], None, None, None
        else:
            hist0, mom0, rm, rv = [row[-D:] for row in res["history"]], res["momentum"], res["run_mean"], res["run_var"]
        res = O.train_from(wl.ops, wl.in_shape, wl.stage_end, t_prev, hist0, mom0, xs[t_prev:t], ys[t_prev:t],
                           st[t_prev:t], lr[t_prev:t], wl.momentum, wl.weight_decay, wl.nesterov, bf16=wl.bf16,
                           dropout_seed=wl.dropout_seed, run_mean=rm, run_var=rv, out_depth=D)
        for s_, row in enumerate(res["history"]):
            out[f"t{t}_s{s_}"] = np.stack(row[D - depth[s_]:]).astype(np.float32)  # versions t-d_s .. t
        out[f"t{t}_momentum"] = res["momentum"].astype(np.float32)
        out[f"t{t}_run_mean"] = res["run_mean"].astype(np.float32)
        out[f"t{t}_run_var"] = res["run_var"].astype(np.float32)
        print(f"states {mode}: t={t} {time.time() - t0:.0f} s, loss {res['losses'][-1]:.6f}", flush=True)
        t_prev = t
    path = os.path.join(HERE, f"resnet20_b128_states_{mode}.npz")
    np.savez_compressed(path, steps=np.array(STATE_STEPS), **out)
    print(f"-> {path} ({os.path.getsize(path) / 2**20:.1f} MiB)", flush=True)


if __name__ == "__main__":
    for m in (sys.argv[1:] or ["fp32", "bf16"]):
        if m in ("fp32", "bf16"):
            make(m)
        elif m.startswith("states_"):
            make_states(m[len("states_"):])
        else:
            make_full(m)
