"""Workload descriptions and seeded synthetic inputs.

This module is the only thing the GPU path and the CPU oracle both consume.
It holds no arithmetic of the method: it describes networks as operation
lists, names the pipeline split and the staleness schedule of each workload,
and draws seeded float32 inputs, labels and initial weights.

Network description (one row of nine int32 per operation; tensor 0 is the
mini-batch, operation i writes tensor i+1):

    kind, in0, in1, cin, cout, k, stride, pad, flags

kind: 1 conv, 2 batch-norm (+ optional residual in1, + optional ReLU),
3 max-pool (k x k, stride, no padding), 4 global average pool, 5 fully
connected, 6 dropout (k = drop probability in units of 2^-24; its mask is a
function of the seed, the operation, the step and the element, so the
backward pass of a mini-batch recomputes the forward's mask).  flags: bit0
bias, bit1 ReLU.  A batch-norm whose residual has
fewer channels or a larger spatial size than its output uses the CIFAR-ResNet
"option A" shortcut (subsample + zero channel padding).

The paper numbers weighted layers 1..L (Sec. 3); a Pipeline Placement Vector
(p_1..p_K) puts a register pair after layer p_i.  ``layer_end[l]`` maps layer
l to one past its last operation (its BN, residual add and pooling included),
which turns a PPV into operation-index stage boundaries.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, List, Sequence

import numpy as np

CONV, BN, MAXPOOL, GAVG, FC, DROPOUT = 1, 2, 3, 4, 5, 6
F_BIAS, F_RELU = 1, 2


def dropout_threshold(p: float) -> int:
    """The dropout op's k field: drop probability p in units of 2^-24."""
    k = int(round(p * (1 << 24)))
    assert 0 < k < (1 << 24), p
    return k


@dataclasses.dataclass
class Workload:
    name: str
    ops: np.ndarray                 # [n_ops, 9] int32
    in_shape: tuple                 # (C, H, W)
    classes: int
    batch: int
    layer_end: List[int]            # layer_end[l] for l = 1..L (index 0 unused)
    stage_end: List[int]            # one past the last op of every stage
    staleness_fn: Callable[[int], List[int]]
    steps: int
    lr: List[float]
    momentum: float = 0.9
    weight_decay: float = 0.0
    nesterov: bool = False
    bf16: bool = False
    seed: int = 0
    input_dist: str = "normal"      # "normal" N(0,1) or "uniform" U[0,1)
    lr_fn: Callable[[int], List[float]] | None = None  # per-step, per-stage rates (default: lr every step)
    dropout_seed: int = 0            # key of the dropout masks (64-bit)

    @property
    def n_stages(self) -> int:
        return len(self.stage_end)

    def lr_at(self, t: int) -> List[float]:
        return list(self.lr_fn(t)) if self.lr_fn is not None else list(self.lr)

    def lr_table(self, steps: int | None = None, t0: int = 0) -> np.ndarray:
        """[T, S] learning rates of steps t0 .. t0+T-1."""
        T = self.steps if steps is None else steps
        return np.array([self.lr_at(t0 + t) for t in range(T)], dtype=np.float64).reshape(T, self.n_stages)

    def staleness(self, steps: int | None = None) -> np.ndarray:
        T = self.steps if steps is None else steps
        return np.array([self.staleness_fn(t) for t in range(T)], dtype=np.int32).reshape(T, self.n_stages)

    def ring_depth(self, steps: int | None = None) -> List[int]:
        st = self.staleness(steps)
        return [int(st[:, s].max()) + 1 for s in range(self.n_stages)]


class _Builder:
    def __init__(self):
        self.ops: List[List[int]] = []
        self.layer_end: List[int] = [0]

    def add(self, kind, in0, cin, cout, k=0, stride=1, pad=0, flags=0, in1=-1) -> int:
        self.ops.append([kind, in0, in1, cin, cout, k, stride, pad, flags])
        return len(self.ops)  # id of the tensor this op writes

    def end_layer(self):
        self.layer_end.append(len(self.ops))

    def desc(self) -> np.ndarray:
        return np.array(self.ops, dtype=np.int32).reshape(-1, 9)


def _stage_end_from_ppv(layer_end: Sequence[int], ppv: Sequence[int], n_ops: int) -> List[int]:
    return [layer_end[p] for p in ppv] + [n_ops]


# ------------------------------------------------------------------ nets ----
def lenet5():
    """LeNet-5 on 1x28x28: conv 6@5x5 pad 2 + ReLU, maxpool 2, conv 16@5x5 +
    ReLU, maxpool 2, fc 400-120-84-10 (ReLU between FCs)."""
    b = _Builder()
    t = b.add(CONV, 0, 1, 6, 5, 1, 2, F_BIAS | F_RELU)
    t = b.add(MAXPOOL, t, 6, 6, 2, 2)
    b.end_layer()
    t = b.add(CONV, t, 6, 16, 5, 1, 0, F_BIAS | F_RELU)
    t = b.add(MAXPOOL, t, 16, 16, 2, 2)
    b.end_layer()
    t = b.add(FC, t, 400, 120, flags=F_BIAS | F_RELU)
    b.end_layer()
    t = b.add(FC, t, 120, 84, flags=F_BIAS | F_RELU)
    b.end_layer()
    b.add(FC, t, 84, 10, flags=F_BIAS)
    b.end_layer()
    return b.desc(), b.layer_end, (1, 28, 28)


def alexnet_cifar():
    """AlexNet-style CIFAR net: conv 64@5x5, pool, conv 192@5x5, pool,
    conv 384/256/256@3x3, fc 4096-4096-10 (5x5 pad 2, 3x3 pad 1, bias, ReLU,
    max-pool 2x2/2)."""
    b = _Builder()
    t = b.add(CONV, 0, 3, 64, 5, 1, 2, F_BIAS | F_RELU)
    t = b.add(MAXPOOL, t, 64, 64, 2, 2)
    b.end_layer()
    t = b.add(CONV, t, 64, 192, 5, 1, 2, F_BIAS | F_RELU)
    t = b.add(MAXPOOL, t, 192, 192, 2, 2)
    b.end_layer()
    for cin, cout in ((192, 384), (384, 256), (256, 256)):
        t = b.add(CONV, t, cin, cout, 3, 1, 1, F_BIAS | F_RELU)
        b.end_layer()
    t = b.add(FC, t, 256 * 8 * 8, 4096, flags=F_BIAS | F_RELU)
    b.end_layer()
    t = b.add(FC, t, 4096, 4096, flags=F_BIAS | F_RELU)
    b.end_layer()
    b.add(FC, t, 4096, 10, flags=F_BIAS)
    b.end_layer()
    return b.desc(), b.layer_end, (3, 32, 32)


def vgg16_bn(dropout: float | None = None):
    """VGG-16 with BN, CIFAR shape: 13 conv 3x3 (no bias) -> BN -> ReLU,
    max-pool 2x2/2 after convs 2, 4, 7, 10, 13, fc 512-10.  With dropout = p:
    dropout(p) after every BN+ReLU that no max-pool follows, and before the
    classifier (App. A names dropout for VGG-16 without placing it)."""
    b = _Builder()
    chans = [64, 64, 128, 128, 256, 256, 256, 512, 512, 512, 512, 512, 512]
    pools = {2, 4, 7, 10, 13}
    t, cin = 0, 3
    for i, c in enumerate(chans, start=1):
        t = b.add(CONV, t, cin, c, 3, 1, 1, 0)
        t = b.add(BN, t, c, c, flags=F_RELU)
        if i in pools:
            t = b.add(MAXPOOL, t, c, c, 2, 2)
        elif dropout is not None:
            t = b.add(DROPOUT, t, c, c, dropout_threshold(dropout))
        b.end_layer()
        cin = c
    if dropout is not None:
        t = b.add(DROPOUT, t, 512, 512, dropout_threshold(dropout))
    b.add(FC, t, 512, 10, flags=F_BIAS)
    b.end_layer()
    return b.desc(), b.layer_end, (3, 32, 32)


def resnet_cifar(depth: int):
    """CIFAR ResNet of depth 6n+2: stem conv 3x3 16 + BN + ReLU, three groups of
    n basic blocks (16/32/64 channels, first block of groups 2 and 3 has
    stride 2), option-A shortcuts, global average pool, fc 64-10 (bias).
    Convs have no bias."""
    assert (depth - 2) % 6 == 0
    n = (depth - 2) // 6
    b = _Builder()
    t = b.add(CONV, 0, 3, 16, 3, 1, 1, 0)
    t = b.add(BN, t, 16, 16, flags=F_RELU)
    b.end_layer()
    cin = 16
    for g, c in enumerate((16, 32, 64)):
        for blk in range(n):
            stride = 2 if (g > 0 and blk == 0) else 1
            x_in = t
            t = b.add(CONV, t, cin, c, 3, stride, 1, 0)
            t = b.add(BN, t, c, c, flags=F_RELU)
            b.end_layer()
            t = b.add(CONV, t, c, c, 3, 1, 1, 0)
            t = b.add(BN, t, c, c, flags=F_RELU, in1=x_in)
            b.end_layer()
            cin = c
    t = b.add(GAVG, t, 64, 64)
    b.add(FC, t, 64, 10, flags=F_BIAS)
    b.end_layer()
    return b.desc(), b.layer_end, (3, 32, 32)


# ------------------------------------------------- learning-rate policies ---
# The schedules of App. A and B, as functions of the step t (one mini-batch).
def lr_step(base: float, milestones: Sequence[int], gamma: float = 0.1) -> Callable[[int], float]:
    """base, multiplied by gamma at every milestone step reached ("decreased by
    10x twice": ResNet and AlexNet)."""
    ms = sorted(int(m) for m in milestones)
    return lambda t: base * gamma ** sum(1 for m in ms if t >= m)


def lr_halving(base: float, period: int) -> Callable[[int], float]:
    """base, halved every `period` steps (VGG-16: every 50 epochs)."""
    return lambda t: base * 0.5 ** (t // period)


def lr_inverse(base: float, gamma: float = 1e-4, power: float = 0.75) -> Callable[[int], float]:
    """The inverse policy named for LeNet-5: base * (1 + gamma t)^(-power)."""
    return lambda t: base * (1.0 + gamma * t) ** (-power)


# Two-partition pipelines of the actual pipelined training (Table 5): the
# register pair after layer p, and the learning rate of BKS_2, the backward
# stage of the first partition (Table 7); the other hyperparameters are those
# of the non-pipelined baseline (App. B: 0.1, x0.1 at epochs 100 and 150,
# momentum 0.9, weight decay 1e-4, batch 128).
TABLE5_PPV = {20: 7, 56: 19, 110: 37, 224: 75, 362: 121}
TABLE7_BKS2_LR = {20: 0.1, 56: 0.01, 110: 0.001, 224: 0.001, 362: 0.001}
CIFAR_STEPS_PER_EPOCH = 391  # 50,000 images in batches of 128, the last one partial


# ------------------------------------------------------------- workloads ----
def _const(d):
    return lambda t: list(d)


def lenet5_workload(batch=16, steps=1, seed=1912):
    ops, le, ins = lenet5()
    return Workload("lenet5", ops, ins, 10, batch, le, [len(ops)], _const([0]), steps, [0.01],
                    seed=seed, input_dist="uniform")


def alexnet_workload(batch=128, steps=20, seed=1913):
    """App. A's AlexNet hyperparameters: rate 0.001, Nesterov momentum 0.9,
    weight decay 0.004 (at rate 0.01 this net without BN diverges on these
    inputs within a few steps)."""
    ops, le, ins = alexnet_cifar()
    se = _stage_end_from_ppv(le, (2,), len(ops))        # split after conv2 (and its pool)
    return Workload("alexnet_cifar", ops, ins, 10, batch, le, se, _const([2, 0]), steps, [0.001, 0.001],
                    weight_decay=0.004, nesterov=True, seed=seed)


def resnet20_workload(batch=128, steps=50, seed=1914, bf16=False):
    ops, le, ins = resnet_cifar(20)
    se = _stage_end_from_ppv(le, (7, 13, 19), len(ops))  # Table 1, ResNet-20 (7,13,19)
    return Workload("resnet20" + ("_bf16" if bf16 else ""), ops, ins, 10, batch, le, se,
                    _const([3, 2, 1, 0]), steps, [0.01] * 4, seed=seed, bf16=bf16)


def vgg16_workload(batch=128, steps=40, n_pipelined=30, seed=1915, dropout=None):
    ops, le, ins = vgg16_bn(dropout)
    se = _stage_end_from_ppv(le, (2, 4, 7), len(ops))    # Table 1, VGG-16 (2,4,7)

    def hybrid(t, n_p=n_pipelined):
        return [3, 2, 1, 0] if t < n_p else [0, 0, 0, 0]
    return Workload("vgg16_bn" + ("_dropout" if dropout is not None else ""), ops, ins, 10, batch, le, se, hybrid,
                    steps, [0.01] * 4, seed=seed, dropout_seed=(seed << 32) | 0x5EED if dropout is not None else 0)


def resnet110_workload(batch=256, steps=50, seed=1916, bf16=True):
    ops, le, ins = resnet_cifar(110)
    blocks = [7, 7, 7, 7, 7, 7, 6, 6]
    ppv = list(np.cumsum(blocks)[:-1] * 2 + 1)          # block b ends at layer 1 + 2b
    se = _stage_end_from_ppv(le, ppv, len(ops))
    return Workload("resnet110" + ("_bf16" if bf16 else ""), ops, ins, 10, batch, le, se,
                    _const([7 - s for s in range(8)]), steps, [0.01] * 8, seed=seed, bf16=bf16)


def resnet_two_partition_workload(depth=20, batch=128, steps=50, n_pipelined=None,
                                  steps_per_epoch=CIFAR_STEPS_PER_EPOCH, seed=1917):
    """ResNet-depth split by one register pair at its Table 5 PPV (two
    partitions, the paper's 4-stage pipeline on 2 devices).  Staleness under
    the cycle schedule with K = 1: d = 2(K - i + 1) = [2, 0].  Hybrid (Sec. 4)
    when n_pipelined is given: d = [0, 0] from that step on (100 of 200 epochs
    in Table 5).  Rates: the baseline's step policy, with the first partition's
    backward stage (BKS_2) starting at its Table 7 rate and decayed alike."""
    ops, le, ins = resnet_cifar(depth)
    se = _stage_end_from_ppv(le, (TABLE5_PPV[depth],), len(ops))

    def stal(t):
        return [2, 0] if n_pipelined is None or t < n_pipelined else [0, 0]

    decay = lr_step(1.0, (100 * steps_per_epoch, 150 * steps_per_epoch))

    def lr_fn(t):
        return [TABLE7_BKS2_LR[depth] * decay(t), 0.1 * decay(t)]

    return Workload(f"resnet{depth}_2part", ops, ins, 10, batch, le, se, stal, steps,
                    [TABLE7_BKS2_LR[depth], 0.1], weight_decay=1e-4, seed=seed, lr_fn=lr_fn)


WORKLOADS = {
    "lenet5": lenet5_workload,
    "alexnet": alexnet_workload,
    "resnet20": resnet20_workload,
    "vgg16": vgg16_workload,
    "resnet110": resnet110_workload,
}


# ------------------------------------------------------------- generators ---
def param_layout(wl: Workload):
    """[(op_index, name, shape, stage, offset_in_stage)] for every parameter
    tensor, in the flat per-stage order (conv: weight, bias; bn: gamma, beta;
    fc: weight, bias)."""
    out = []
    stage_of = np.zeros(len(wl.ops), dtype=int)
    prev = 0
    for s, e in enumerate(wl.stage_end):
        stage_of[prev:e] = s
        prev = e
    off = [0] * wl.n_stages
    for i, o in enumerate(wl.ops):
        kind, _, _, cin, cout, k, _, _, flags = (int(v) for v in o)
        s = int(stage_of[i])
        items = []
        if kind == CONV:
            items.append(("weight", (cout, cin, k, k)))
            if flags & F_BIAS:
                items.append(("bias", (cout,)))
        elif kind == BN:
            items += [("gamma", (cin,)), ("beta", (cin,))]
        elif kind == FC:
            items.append(("weight", (cout, cin)))
            if flags & F_BIAS:
                items.append(("bias", (cout,)))
        for name, shape in items:
            out.append((i, name, shape, s, off[s]))
            off[s] += int(np.prod(shape))
    return out, off


def init_params(wl: Workload) -> np.ndarray:
    """Initial weights W^(0), float32, stages concatenated.  Conv and FC
    weights: uniform(-sqrt(6/fan_in), +sqrt(6/fan_in)) (Kaiming uniform),
    biases 0, BN gamma 1 and beta 0."""
    layout, counts = param_layout(wl)
    rng = np.random.Generator(np.random.PCG64([wl.seed, 0]))
    stage_base = np.concatenate([[0], np.cumsum(counts)])
    flat = np.zeros(int(stage_base[-1]), dtype=np.float32)
    for _, name, shape, s, off in layout:
        n = int(np.prod(shape))
        base = int(stage_base[s]) + off
        if name == "weight":
            fan_in = int(np.prod(shape[1:]))
            bound = np.sqrt(6.0 / fan_in)
            flat[base:base + n] = rng.uniform(-bound, bound, size=n).astype(np.float32)
        elif name == "gamma":
            flat[base:base + n] = 1.0
        # bias, beta: 0
    return flat


def batch(wl: Workload, t: int, batch_size: int | None = None):
    """Mini-batch t: (x float32 [N,C,H,W], labels int32 [N])."""
    N = wl.batch if batch_size is None else batch_size
    rng = np.random.Generator(np.random.PCG64([wl.seed, 1, t]))
    shape = (N,) + tuple(wl.in_shape)
    if wl.input_dist == "uniform":
        x = rng.random(size=shape, dtype=np.float32)
    else:
        x = rng.standard_normal(size=shape, dtype=np.float32)
    labels = rng.integers(0, wl.classes, size=N, dtype=np.int32)
    return x, labels


def batches(wl: Workload, T: int, batch_size: int | None = None):
    xs, ys = zip(*(batch(wl, t, batch_size) for t in range(T)))
    return np.stack(xs), np.stack(ys)
