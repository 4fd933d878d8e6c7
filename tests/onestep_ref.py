"""Reference side of the one-step comparisons (CPU only): checkpoints of
the stale-weight schedule at step t (the oracle's own trajectory, or a
seeded synthetic state), one step of the oracle from such a state, the same
step in torch autograd, and the distances the comparisons report.

A checkpoint holds what step t of the schedule reads (Sec. 3): the ring
window W_s^(t-D_s+1) .. W_s^(t) of every stage, the momentum, and the BN
running statistics."""
import os

import numpy as np
import torch

from paper_1912_12675_amd import synth
from tests import torch_ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


class State:
    """Checkpoint at step t: window[s] maps version -> float32 vector of
    stage s (versions max(0, t-D_s+1) .. t), momentum, running statistics."""

    def __init__(self, t, window, momentum, run_mean, run_var):
        self.t, self.window, self.momentum, self.run_mean, self.run_var = t, window, momentum, run_mean, run_var

    def version(self, s, v):
        return self.window[s][v]


def _counts(oracle, wl):
    return [int(c) for c in oracle.param_counts(wl.ops, wl.in_shape, 1, wl.stage_end)]


def _split(flat, counts):
    return np.split(np.asarray(flat), np.cumsum(counts)[:-1])


def _n_bn(wl):
    return int(sum(int(o[4]) for o in wl.ops if int(o[0]) == synth.BN))


def resnet20_state(oracle, wl, t):
    counts = _counts(oracle, wl)
    depth = wl.ring_depth()
    p0 = synth.init_params(wl)
    nbn = _n_bn(wl)
    if t == 0:
        return State(0, [{0: v} for v in _split(p0, counts)], np.zeros(sum(counts), np.float32),
                     np.zeros(nbn, np.float32), np.ones(nbn, np.float32))
    if t == 1:  # the oracle's first step, rounded to float32 like a stored state
        xs, ys = synth.batches(wl, 1)
        r = oracle.train_from(wl.ops, wl.in_shape, wl.stage_end, 0, [[v] for v in _split(p0, counts)], None, xs, ys,
                              wl.staleness(1), wl.lr_table(1), wl.momentum, wl.weight_decay, wl.nesterov,
                              bf16=wl.bf16, out_depth=2)
        win = [{0: p0s, 1: r["history"][s][1].astype(np.float32)} for s, p0s in enumerate(_split(p0, counts))]
        return State(1, win, r["momentum"].astype(np.float32), r["run_mean"].astype(np.float32),
                     r["run_var"].astype(np.float32))
    mode = "bf16" if wl.bf16 else "fp32"
    path = os.path.join(GOLDEN, f"resnet20_b128_states_{mode}.npz")
    assert os.path.exists(path), f"missing {path} (python tests/golden/make_golden.py states_{mode})"
    g = np.load(path)
    win = []
    for s in range(len(counts)):
        vs = g[f"t{t}_s{s}"]
        assert vs.shape == (depth[s], counts[s])
        win.append({t - depth[s] + 1 + k: vs[k] for k in range(depth[s])})
    return State(t, win, g[f"t{t}_momentum"], g[f"t{t}_run_mean"], g[f"t{t}_run_var"])


def synthetic_state(oracle, wl, t, seed):
    """Seeded checkpoint at step t: version v of stage s is W^(0) moved by
    1e-3 * N(0,1) * (|W^(0)| + 1e-2) (a fresh draw per version), the momentum
    1e-2 * N(0,1) * (|W^(0)| + 1e-2), running statistics mean 0 / var 1."""
    counts = _counts(oracle, wl)
    depth = wl.ring_depth(t + 1)
    rng = np.random.Generator(np.random.PCG64([seed, t]))
    p0 = synth.init_params(wl)
    win = []
    for s, p in enumerate(_split(p0, counts)):
        scale = np.abs(p) + np.float32(1e-2)
        win.append({v: (p + np.float32(1e-3) * rng.standard_normal(p.size, dtype=np.float32) * scale)
                    for v in range(max(0, t - depth[s] + 1), t + 1)})
    mom = (np.float32(1e-2) * rng.standard_normal(p0.size, dtype=np.float32) * (np.abs(p0) + np.float32(1e-2)))
    nbn = _n_bn(wl)
    return State(t, win, mom.astype(np.float32), np.zeros(nbn, np.float32), np.ones(nbn, np.float32))


def oracle_step(oracle, wl, state):
    t = state.t
    D = max(len(w) for w in state.window)
    hist0 = [[w.get(v) for v in range(t - D + 1, t + 1)] for w in state.window]
    hist0 = [[None if a is None else a.astype(np.float64) for a in row] for row in hist0]
    x, y = synth.batch(wl, t)
    st = wl.staleness(t + 1)[t:t + 1]
    nbn = _n_bn(wl)
    r = oracle.train_from(wl.ops, wl.in_shape, wl.stage_end, t, hist0, state.momentum.astype(np.float64), x[None],
                          y[None], st, wl.lr_table(1, t0=t), wl.momentum, wl.weight_decay, wl.nesterov, bf16=wl.bf16,
                          dropout_seed=wl.dropout_seed,
                          run_mean=state.run_mean.astype(np.float64) if nbn else None,
                          run_var=state.run_var.astype(np.float64) if nbn else None)
    return dict(versions=r["versions"][0], grad=r["grad"], momentum=r["momentum"], params=r["params"],
                loss=float(r["losses"][0]))


def ulp_move(x, seed):
    """x moved one float32 ulp up or down element by element (seeded signs)."""
    up = np.random.Generator(np.random.PCG64(seed)).random(x.shape) < 0.5
    return np.where(up, np.nextafter(x, np.float32(np.inf)), np.nextafter(x, np.float32(-np.inf))).astype(np.float32)


def torch_step(wl, state, x=None, dtype=torch.float32, decisions=None):
    """The same step in torch (CPU, float32 unless dtype says otherwise),
    bf16-rounded product operands in bf16 mode; x replaces the step's
    mini-batch when given; decisions: ReLU decisions to record or to take
    (torch_ref._relu)."""
    t = state.t
    st = wl.staleness(t + 1)[t]
    wfor = [w[max(0, t - int(st[s]))] for s, w in enumerate(state.window)]
    wcur = [w[t] for w in state.window]
    xb, y = synth.batch(wl, t)
    return torch_ref.stale_step_from(wl.ops, wl.stage_end, wfor, wcur, state.momentum, xb if x is None else x, y,
                                     wl.lr_at(t), wl.momentum, wl.weight_decay, wl.nesterov, dtype=dtype,
                                     bf16=wl.bf16, dropout_key=(wl.dropout_seed, t), decisions=decisions)


def rel(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def distances(wl, got, ref, w_t):
    """Distances of `got` from the oracle's `ref` (w_t: W^(t), float32 values)."""
    layout, counts = synth.param_layout(wl)
    base = np.concatenate([[0], np.cumsum(counts)])
    per = {}
    for op, name, shape, s, off in layout:
        i0 = int(base[s]) + off
        sl = slice(i0, i0 + int(np.prod(shape)))
        per[f"op {op} {name}{tuple(shape)}"] = rel(got["grad"][sl], ref["grad"][sl])
    return dict(grad=rel(got["grad"], ref["grad"]), per=per, momentum=rel(got["momentum"], ref["momentum"]),
                update=rel(got["params"] - w_t, ref["params"] - w_t),
                loss=abs(got["loss"] - ref["loss"]) / abs(ref["loss"]))
