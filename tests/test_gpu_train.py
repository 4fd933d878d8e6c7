"""End-to-end GPU parity of the stale-weight training path (psw_stage_step)
against the oracle: parameters after N steps, per-step losses, and the
weight-version table.

Bar: ||gpu - oracle||_2 / ||oracle||_2 <= 1e-4 (fp32) or 2e-2 (bf16 mode)
over the whole parameter vector and for every tensor with a non-zero
initial value, widened to 4x the spread of an independent computation where
a run amplifies rounding (see test_train_parity); versions equal as
integers.  The small cases
run the oracle live at sizes it finishes in seconds; the full-size ResNet-20
case (batch 128, 50 steps, the configuration bench.py times) compares with
the oracle's stored result (tests/golden/make_golden.py)."""
import os

import numpy as np
import pytest
import torch

from paper_1912_12675_amd import synth
from tests import torch_ref
from tests.test_abi import conv_residual_workload

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def P():
    from paper_1912_12675_amd import psw
    psw.lib()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return psw


def gpu_train(P, wl, T, batch=None, net=None, t0=0, stash=False):
    N = wl.batch if batch is None else batch
    st = wl.staleness(T)
    if net is None:
        net = P.Net(wl.ops, N, wl.in_shape, wl.stage_end, wl.ring_depth(T), bf16=wl.bf16)
        net.load_params(synth.init_params(wl))
        net.set_dropout_seed(wl.dropout_seed)
        if stash:
            net.set_weight_stashing(True)
    losses, versions = [], []
    for t in range(t0, T):
        x, y = synth.batch(wl, t, N)
        ver = net.step(t, st[t], wl.lr_at(t), torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), wl.momentum,
                       wl.weight_decay, wl.nesterov)
        losses.append(float(net.loss.item()))
        versions.append(ver)
    torch.cuda.synchronize()
    return net, np.array(losses), np.array(versions)


def oracle_train(oracle, wl, T, batch=None, stash=False):
    N = wl.batch if batch is None else batch
    xs, ys = synth.batches(wl, T, N)
    return oracle.train(wl.ops, wl.in_shape, wl.stage_end, synth.init_params(wl), xs, ys, wl.staleness(T), wl.lr_table(T),
                        wl.momentum, wl.weight_decay, wl.nesterov, bf16=wl.bf16, stash=stash,
                        dropout_seed=wl.dropout_seed)


def deviations(wl, flat, losses, ref_flat, ref_losses, p0):
    """(whole-vector params rel-L2, {tensor: rel-L2} for tensors with a
    non-zero initial value, max loss rel, update rel-L2)."""
    layout, counts = synth.param_layout(wl)
    base = np.concatenate([[0], np.cumsum(counts)])
    glob = np.linalg.norm(flat - ref_flat) / np.linalg.norm(ref_flat)
    upd = np.linalg.norm((flat - p0) - (ref_flat - p0)) / max(np.linalg.norm(ref_flat - p0), 1e-30)
    per = {}
    for op, name, shape, s, off in layout:
        n = int(np.prod(shape))
        i0 = int(base[s]) + off
        if np.linalg.norm(p0[i0:i0 + n]) > 0.0:
            per[f"op {op} {name}{shape}"] = np.linalg.norm(flat[i0:i0 + n] - ref_flat[i0:i0 + n]) / \
                np.linalg.norm(ref_flat[i0:i0 + n])
    lrel = np.abs(np.asarray(losses) - ref_losses).max() / np.abs(ref_losses).max()
    return glob, per, lrel, upd


def reference_spread(oracle, wl, T, batch, xs, ys, stash=False):
    """Independent computations at the GPU's precision, to measure how far
    such a computation lands from the oracle on this run: the stale schedule
    written with torch autograd in float32 (CPU) -- in bf16 mode with both
    operands of every product rounded to bfloat16 -- on the inputs and on
    the inputs moved one float32 ulp up and down.  Returns a list of
    (params, losses)."""
    p0 = synth.init_params(wl)
    up = np.nextafter(xs, np.inf, dtype=np.float32)
    down = np.nextafter(xs, -np.inf, dtype=np.float32)
    out = []
    for inp in (xs, up, down):
        p, l, _ = torch_ref.train_stale(wl.ops, wl.stage_end, p0, inp, ys, wl.staleness(T), wl.lr_table(T), wl.momentum,
                                        wl.weight_decay, dtype=torch.float32, stash=stash,
                                        dropout_seed=wl.dropout_seed, bf16=wl.bf16, nesterov=wl.nesterov)
        out.append((p, l))
    return out


CASES = [
    # (workload factory, batch, steps)
    ("lenet5", lambda: synth.lenet5_workload(), 16, 1),
    ("resnet20_b8", lambda: synth.resnet20_workload(batch=8), 8, 10),
    # batch 6: the folded BN merges' per-thread tile counts do not divide
    # evenly at any layer (24, 12 and 6 tiles over 16, 16 and 8 threads), and
    # the 8x8 weight gradients take the unsplit path (6 is not a multiple of 4)
    ("resnet20_b6", lambda: synth.resnet20_workload(batch=6), 6, 8),
    ("resnet20_bf16_b8", lambda: synth.resnet20_workload(batch=8, bf16=True), 8, 6),
    ("alexnet_b4", lambda: synth.alexnet_workload(batch=4), 4, 4),
    ("vgg16_hybrid_b16", lambda: synth.vgg16_workload(batch=16, n_pipelined=3), 16, 5),
    ("resnet110_bf16_b8", lambda: synth.resnet110_workload(batch=8), 8, 3),
    # Table 5's two-partition ResNet-56 (PPV (19), d = [2, 0], BKS_2 rate of
    # Table 7, weight decay 1e-4) with its step policy compressed so that both
    # decays fall inside the run, then the hybrid switch
    ("resnet56_2part_b8", lambda: synth.resnet_two_partition_workload(56, batch=8, n_pipelined=4,
                                                                       steps_per_epoch=0.02), 8, 6),
    # VGG-16 with dropout (Philox masks, recomputed by each step's backward).
    # At batch 8 this run is chaotic for every float32 implementation: moving
    # the inputs by one ulp moves the GPU's result from 1.9e-2 to 4e-7 of the
    # oracle (a max-pool / ReLU near-tie decided the other way), so the case
    # runs at batch 16 like the plain VGG-16 case.
    ("vgg16_dropout_b16", lambda: synth.vgg16_workload(batch=16, n_pipelined=3, dropout=0.4), 16, 5),
    # a residual BN that adds its block conv's own input (x -> conv ->
    # BN(+x)): its backward is not folded into that conv's backward-data
    # kernel, which reads the gradient the fold would write
    ("conv_residual_b4", lambda: conv_residual_workload(batch=4), 4, 4),
]


STASH_CASES = [
    ("resnet20_b8_stash", lambda: synth.resnet20_workload(batch=8), 8, 10),
    ("alexnet_b4_stash", lambda: synth.alexnet_workload(batch=4), 4, 4),
]


@pytest.mark.parametrize("name,factory,batch,T,stash", [c + (False,) for c in CASES] + [c + (True,) for c in STASH_CASES],
                         ids=[c[0] for c in CASES] + [c[0] for c in STASH_CASES])
def test_train_parity(P, oracle, name, factory, batch, T, stash):
    """Bar: max(target, 4 x reference spread) for the whole parameter
    vector, for every tensor with a non-zero initial value, and for the
    losses; the target is 1e-4 (fp32) / 2e-2 (bf16).  The spread
    (the largest deviation among the reference_spread samples: torch float32,
    with bf16-rounded product operands in bf16 mode) measures how
    much this particular run amplifies
    rounding-level differences: ReLU-sign and max-pool decisions taken near
    zero, and in bf16 mode operand roundings, flip between any two
    implementations that do not share every intermediate bit.  In VGG-16 one
    such flip (a max-pool near-tie) already moves every gradient below it by
    1e-3..2e-3 in a single step, for torch float32 as for the GPU.

    The *_stash cases run the comparison scheme (weight stashing: data
    gradients with the forward's version) against the oracle's stash mode."""
    print(f"train parity {name}: batch {batch}, {T} steps", flush=True)
    wl = factory()
    net, losses, versions = gpu_train(P, wl, T, batch, stash=stash)
    ref = oracle_train(oracle, wl, T, batch, stash=stash)
    xs, ys = synth.batches(wl, T, batch)
    p0 = synth.init_params(wl).astype(np.float64)
    got = net.params(T).double().numpy()
    g_glob, g_per, g_loss, g_upd = deviations(wl, got, losses, ref["params"], ref["losses"], p0)
    s_glob = s_loss = s_upd = 0.0
    s_per = {}
    for sp_p, sp_l in reference_spread(oracle, wl, T, batch, xs, ys, stash=stash):
        a, b, c, d = deviations(wl, sp_p, sp_l, ref["params"], ref["losses"], p0)
        s_glob, s_loss, s_upd = max(s_glob, a), max(s_loss, c), max(s_upd, d)
        s_per = {k: max(s_per.get(k, 0.0), v) for k, v in b.items()}
    bar = 2e-2 if wl.bf16 else 1e-4
    worst = max(g_per, key=g_per.get)
    print(f"{name}: gpu params {g_glob:.2e} update {g_upd:.2e} loss {g_loss:.2e} worst tensor {g_per[worst]:.2e} "
          f"({worst}) | reference spread params {s_glob:.2e} update {s_upd:.2e} loss {s_loss:.2e} "
          f"tensor {s_per[worst]:.2e}", flush=True)
    np.testing.assert_array_equal(versions, ref["versions"])
    np.testing.assert_array_equal(versions, np.maximum(0, np.arange(T)[:, None] - wl.staleness(T)))
    assert g_glob <= max(bar, 4 * s_glob), f"params rel-L2 {g_glob:.3e}"
    # a flipped decision moves parameters and loss alike: the loss is held to
    # the larger of the two spreads
    assert g_loss <= max(bar, 4 * max(s_loss, s_glob)), f"loss rel {g_loss:.3e}"
    for k, v in g_per.items():
        assert v <= max(bar, 4 * s_per[k]), f"{k}: rel-L2 {v:.3e} (spread {s_per[k]:.3e})"
    # the stale schedule changes the result (it is not plain SGD in disguise)
    if T > 1 and wl.staleness(T).max() > 0:
        assert np.abs(ref["params"] - p0).max() > 0


@pytest.mark.parametrize("mode", ["fp32", "bf16"])
def test_resnet20_full_size_50_steps(P, mode):
    """ResNet-20, batch 128, PPV (7,13,19), staleness [3,2,1,0], 50 steps:
    the configuration the benchmark times, against the stored oracle run.

    This is a trajectory check, not the parity bar: over 50 steps rounding
    differences are amplified (an independent float32 implementation, torch
    on the CPU with the same schedule, ends 3.7e-3 from the float64 oracle
    in parameters, i.e. 15% of the 50-step update), so the tight comparison
    is one step from identical states (tests/test_gpu_onestep.py).  Here:
    versions exact; losses within 2e-3 (fp32) / 2e-2 (bf16); and the
    parameters' update W^(50) - W^(0) within 0.3 (fp32) / 0.6 (bf16) of the
    oracle's update in rel-L2 -- about twice the float32 spread, and far
    below the 1.0 of a run that applied no update or the wrong one."""
    path = os.path.join(GOLDEN, f"resnet20_b128_50steps_{mode}.npz")
    assert os.path.exists(path), f"missing {path} (python tests/golden/make_golden.py)"
    g = np.load(path)
    wl = synth.resnet20_workload(bf16=(mode == "bf16"))
    print(f"resnet20 b128 50 steps {mode}", flush=True)
    net, losses, versions = gpu_train(P, wl, wl.steps)
    p0 = synth.init_params(wl).astype(np.float64)
    ref = p0 + g["delta"].astype(np.float64)
    got = net.params(wl.steps).double().numpy()
    glob = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    upd = np.linalg.norm((got - p0) - (ref - p0)) / np.linalg.norm(ref - p0)
    lrel = np.abs(losses - g["losses"]).max() / np.abs(g["losses"]).max()
    print(f"full size {mode}: params rel-L2 {glob:.3e}, update rel-L2 {upd:.3e}, loss max rel {lrel:.3e}", flush=True)
    np.testing.assert_array_equal(versions, g["versions"])
    utol, ltol = (0.6, 2e-2) if wl.bf16 else (0.3, 2e-3)
    assert upd <= utol, f"update rel-L2 {upd:.3e} > {utol}"
    assert lrel <= ltol, f"loss max rel {lrel:.3e} > {ltol}"


def test_runs_are_bit_identical(P):
    wl = synth.resnet20_workload(batch=16)
    a, la, _ = gpu_train(P, wl, 4, 16)
    b, lb, _ = gpu_train(P, wl, 4, 16)
    assert torch.equal(a.params(4), b.params(4))
    np.testing.assert_array_equal(la, lb)


def test_resume_is_bit_identical(P):
    """Checkpoint after 3 steps (ring, momentum, running statistics), resume
    in a new net with psw_net_set_step, continue: same result as an
    uninterrupted run."""
    wl = synth.resnet20_workload(batch=8)
    full, lf, _ = gpu_train(P, wl, 6, 8)
    part, _, _ = gpu_train(P, wl, 3, 8)
    ck = {k: getattr(part, k).clone() for k in ("ring", "momentum", "run_mean", "run_var")}
    net = P.Net(wl.ops, 8, wl.in_shape, wl.stage_end, wl.ring_depth(6), bf16=False)
    for k, v in ck.items():
        getattr(net, k).copy_(v)
    net.set_step(3)
    net, lr_, _ = gpu_train(P, wl, 6, 8, net=net, t0=3)
    assert torch.equal(net.params(6), full.params(6))
    np.testing.assert_array_equal(lr_, lf[3:])
    assert torch.equal(net.run_mean, full.run_mean)


def test_step_order_enforced(P):
    wl = synth.resnet20_workload(batch=2)
    net = P.Net(wl.ops, 2, wl.in_shape, wl.stage_end, wl.ring_depth(), bf16=False)
    x, y = synth.batch(wl, 0, 2)
    with pytest.raises(P.PswError) as e:
        net.step(1, [0, 0, 0, 0], wl.lr, torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda())
    assert e.value.code == -5
    with pytest.raises(P.PswError) as e:
        net.step(0, [4, 0, 0, 0], wl.lr, torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda())
    assert e.value.code == -4


# ---- pipelined execution (psw_pipeline_run) -------------------------------
def _sequential(P, wl, N, st, lr, stash=False):
    net = P.Net(wl.ops, N, wl.in_shape, wl.stage_end, [int(st[:, s].max()) + 1 for s in range(st.shape[1])],
                bf16=wl.bf16)
    net.load_params(synth.init_params(wl))
    net.set_weight_stashing(stash)
    net.set_dropout_seed(wl.dropout_seed)
    losses, versions = [], []
    for t in range(st.shape[0]):
        x, y = synth.batch(wl, t, N)
        lr_t = lr[t] if np.ndim(lr) == 2 else lr
        versions.append(net.step(t, st[t], lr_t, torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), wl.momentum,
                                 wl.weight_decay, wl.nesterov))
        losses.append(float(net.loss.item()))
    torch.cuda.synchronize()
    return net, np.array(losses, dtype=np.float32), np.array(versions)


def _pipelined(P, wl, N, st, lr, chunks, stash=False, step_sets=3):
    T = st.shape[0]
    net = P.Net(wl.ops, N, wl.in_shape, wl.stage_end, [int(st[:, s].max()) + 1 for s in range(st.shape[1])],
                bf16=wl.bf16, step_sets=step_sets)
    net.load_params(synth.init_params(wl))
    net.set_weight_stashing(stash)
    net.set_dropout_seed(wl.dropout_seed)
    xs, ys = synth.batches(wl, T, N)
    xs, ys = torch.from_numpy(xs).cuda(), torch.from_numpy(ys).cuda()
    losses = torch.zeros(T, dtype=torch.float32, device="cuda")
    versions = []
    t0 = 0
    for n in chunks:  # consecutive runs continue the same schedule
        lr_n = lr[t0:t0 + n] if np.ndim(lr) == 2 else lr
        versions.append(net.pipeline_run(t0, st[t0:t0 + n], lr_n, xs[t0:t0 + n], ys[t0:t0 + n], losses[t0:t0 + n],
                                         wl.momentum, wl.weight_decay, wl.nesterov))
        t0 += n
    assert t0 == T
    torch.cuda.synchronize()
    return net, losses.cpu().numpy(), np.concatenate(versions)


def _table(rows, T, S):
    return np.array([rows(t) for t in range(T)], dtype=np.int32).reshape(T, S)


def _mlp_workload(batch=8):
    """Three FC stages and no convolution: every stage is updated on the
    chain's own stream, and the weight stream has no work of its own."""
    b = synth._Builder()
    t = b.add(synth.FC, 0, 784, 64, flags=synth.F_BIAS | synth.F_RELU)
    b.end_layer()
    t = b.add(synth.FC, t, 64, 32, flags=synth.F_BIAS | synth.F_RELU)
    b.end_layer()
    b.add(synth.FC, t, 32, 10, flags=synth.F_BIAS)
    b.end_layer()
    return synth.Workload("mlp", b.desc(), (1, 28, 28), 10, batch, b.layer_end, [1, 2, 3],
                          lambda t: [2, 1, 0], 6, [0.01] * 3, seed=1917)


PIPE_CASES = [
    # name, workload, batch, staleness table (t -> per-stage d), steps, chunks
    ("resnet20_stale", lambda: synth.resnet20_workload(batch=8), 8, lambda t: [3, 2, 1, 0], 8, [8]),
    ("resnet20_paper_d", lambda: synth.resnet20_workload(batch=8), 8, lambda t: [6, 4, 2, 0], 9, [4, 5]),
    ("resnet20_hybrid", lambda: synth.resnet20_workload(batch=8), 8,
     lambda t: [3, 2, 1, 0] if t < 4 else [0, 0, 0, 0], 7, [7]),
    ("resnet20_sgd", lambda: synth.resnet20_workload(batch=8), 8, lambda t: [0, 0, 0, 0], 4, [4]),
    ("resnet20_bf16", lambda: synth.resnet20_workload(batch=8, bf16=True), 8, lambda t: [3, 2, 1, 0], 5, [2, 3]),
    ("alexnet", lambda: synth.alexnet_workload(batch=4), 4, lambda t: [2, 0], 5, [5]),
    ("vgg16_hybrid", lambda: synth.vgg16_workload(batch=8, n_pipelined=3), 8, None, 5, [5]),
    ("resnet20_stash", lambda: synth.resnet20_workload(batch=8), 8, lambda t: [3, 2, 1, 0], 8, [3, 5]),
    ("vgg16_dropout", lambda: synth.vgg16_workload(batch=8, n_pipelined=3, dropout=0.4), 8, None, 5, [2, 3]),
    # eight stages, ring depths 8..1, bf16 products: the deepest ring
    ("resnet110_bf16", lambda: synth.resnet110_workload(batch=4), 4, None, 11, [9, 2]),
    # Table 5's two-partition ResNet-56 with its hybrid switch
    ("resnet56_2part", lambda: synth.resnet_two_partition_workload(56, batch=4, n_pipelined=5,
                                                                    steps_per_epoch=0.03), 4, None, 8, [3, 5]),
    # no convolution anywhere: the step sets are freed through the chain's end
    ("mlp_conv_free", lambda: _mlp_workload(batch=8), 8, None, 9, [9]),
    # uneven tile counts in the folded BN merges (see the batch-6 parity case)
    ("resnet20_b6", lambda: synth.resnet20_workload(batch=6), 6, lambda t: [3, 2, 1, 0], 7, [3, 4]),
]


@pytest.mark.parametrize("name,factory,N,rows,T,chunks", PIPE_CASES, ids=[c[0] for c in PIPE_CASES])
def test_pipeline_run_equals_stage_steps(P, name, factory, N, rows, T, chunks):
    """The pipelined run reorders work across streams only where the
    schedule's dependencies allow it, so it must reproduce the per-step calls
    bit for bit: parameters of the final version, momentum, running
    statistics, every loss and the versions table."""
    wl = factory()
    st = wl.staleness(T) if rows is None else _table(rows, T, len(wl.stage_end))
    stash = name.endswith("_stash")
    a, la, va = _sequential(P, wl, N, st, wl.lr_table(T), stash)
    b, lb, vb = _pipelined(P, wl, N, st, wl.lr_table(T), chunks, stash)
    np.testing.assert_array_equal(va, vb)
    np.testing.assert_array_equal(la, lb)
    assert torch.equal(a.params(T), b.params(T))
    assert torch.equal(a.momentum, b.momentum)
    assert torch.equal(a.run_mean, b.run_mean) and torch.equal(a.run_var, b.run_var)
    print(f"{name}: {T} steps bit-identical, last loss {lb[-1]:.5f}")


def test_pipeline_with_two_step_sets_equals_stage_steps(P):
    """The pipelined run with one step set less (the forward pass of step t
    waits for the weight stream's step t-2): still the per-step result bit
    for bit, over enough steps for the two sets to alternate many times."""
    wl = synth.resnet20_workload(batch=8)
    T = 14
    st = wl.staleness(T)
    a, la, va = _sequential(P, wl, 8, st, wl.lr)
    b, lb, vb = _pipelined(P, wl, 8, st, wl.lr, [5, 9], step_sets=2)
    assert b.step_sets == 2 and b.step2 is not None
    np.testing.assert_array_equal(va, vb)
    np.testing.assert_array_equal(la, lb)
    assert torch.equal(a.params(T), b.params(T))
    assert torch.equal(a.momentum, b.momentum)
    assert torch.equal(a.run_mean, b.run_mean) and torch.equal(a.run_var, b.run_var)


@pytest.mark.parametrize("batch,bf16,T", [(8, False, 8), (8, True, 8), (128, False, 3), (128, True, 3)])
def test_bn_on_load_is_bit_identical(P, batch, bf16, T):
    """The BNs that their consumer conv applies while loading (forward and
    weight gradient, from the BN's input and saved scale / shift) against
    the same net with every BN output stored by its own kernel: the same
    fused multiply-add and ReLU on the same values, so the pipelined run's
    losses, parameters, momentum and running statistics agree bit for bit
    (batch 128: the full-size launch configurations)."""
    wl = synth.resnet20_workload(batch=batch, bf16=bf16)
    st = wl.staleness(T)
    runs = []
    for on in (False, True):
        net = P.Net(wl.ops, batch, wl.in_shape, wl.stage_end, wl.ring_depth(T), bf16=bf16)
        net.set_bn_on_load(on)
        assert all(net.tensor_stored(k) for k in range(1, len(wl.ops) + 1)) != on
        net.load_params(synth.init_params(wl))
        xs, ys = synth.batches(wl, T, batch)
        losses = torch.zeros(T, dtype=torch.float32, device="cuda")
        net.pipeline_run(0, st, wl.lr, torch.from_numpy(xs).cuda(), torch.from_numpy(ys).cuda(), losses, wl.momentum)
        torch.cuda.synchronize()
        runs.append((net, losses.cpu().numpy()))
    (a, la), (b, lb) = runs
    np.testing.assert_array_equal(la, lb)
    assert torch.equal(a.params(T), b.params(T))
    assert torch.equal(a.momentum, b.momentum)
    assert torch.equal(a.run_mean, b.run_mean) and torch.equal(a.run_var, b.run_var)


def test_pipeline_after_stage_steps(P):
    """Per-step calls, then a pipelined run from the next step: same as
    per-step calls throughout."""
    wl = synth.resnet20_workload(batch=8)
    st = _table(lambda t: [3, 2, 1, 0], 6, 4)
    a, la, _ = _sequential(P, wl, 8, st, wl.lr)
    net = P.Net(wl.ops, 8, wl.in_shape, wl.stage_end, [4, 3, 2, 1], bf16=False)
    net.load_params(synth.init_params(wl))
    for t in range(2):
        x, y = synth.batch(wl, t, 8)
        net.step(t, st[t], wl.lr, torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), wl.momentum)
    xs, ys = synth.batches(wl, 6, 8)
    losses = torch.zeros(4, device="cuda")
    net.pipeline_run(2, st[2:], wl.lr, torch.from_numpy(xs[2:]).cuda(), torch.from_numpy(ys[2:]).cuda(), losses,
                     wl.momentum)
    torch.cuda.synchronize()
    assert torch.equal(a.params(6), net.params(6))
    np.testing.assert_array_equal(la[2:], losses.cpu().numpy())


def test_graph_replays_equal_stage_steps(P):
    """A pipelined run captured into a HIP graph (12 steps = the period of
    the ring slots [4,3,2,1] and of the two step sets) and replayed three
    times, with eager work and synchronisations between the replays: after
    every replay the parameters, losses, momentum and running statistics
    equal those of one psw_stage_step call per step."""
    wl = synth.resnet20_workload(batch=8)
    N, fill, per, reps = 8, 3, 12, 3
    T = fill + per * reps
    bidx = [t if t < fill else fill + (t - fill) % per for t in range(T)]
    st = _table(lambda t: [3, 2, 1, 0], T, 4)
    # reference: per-step calls
    ref = P.Net(wl.ops, N, wl.in_shape, wl.stage_end, [4, 3, 2, 1])
    ref.load_params(synth.init_params(wl))
    ref_losses, ref_params = [], {}
    for t in range(T):
        x, y = synth.batch(wl, bidx[t], N)
        ref.step(t, st[t], wl.lr, torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), wl.momentum)
        ref_losses.append(float(ref.loss.item()))
        if t + 1 >= fill and (t + 1 - fill) % per == 0:
            ref_params[t + 1] = ref.params(t + 1).clone()
    # pipeline fill eagerly, then the graph
    net = P.Net(wl.ops, N, wl.in_shape, wl.stage_end, [4, 3, 2, 1])
    net.load_params(synth.init_params(wl))
    xs, ys = synth.batches(wl, fill + per, N)
    xs, ys = torch.from_numpy(xs).cuda(), torch.from_numpy(ys).cuda()
    fill_losses = torch.zeros(fill, device="cuda")
    net.pipeline_run(0, st[:fill], wl.lr, xs[:fill], ys[:fill], fill_losses, wl.momentum)
    losses = torch.zeros(per, device="cuda")
    graph = net.capture(st[fill:fill + per], wl.lr, xs[fill:], ys[fill:], losses, wl.momentum)
    torch.cuda.synchronize()
    assert torch.equal(net.params(fill), ref_params[fill])
    for k in range(reps):
        graph.launch()
        torch.cuda.synchronize()
        t1 = fill + per * (k + 1)
        assert torch.equal(net.params(t1), ref_params[t1]), f"replay {k}"
        np.testing.assert_array_equal(losses.cpu().numpy(), np.array(ref_losses[t1 - per:t1], dtype=np.float32))
        _ = (net.ring.sum() + losses.sum()).item()  # eager work between replays
    assert torch.equal(net.momentum, ref.momentum)
    assert torch.equal(net.run_mean, ref.run_mean) and torch.equal(net.run_var, ref.run_var)


def test_graph_capture_rejects_fill_and_bad_length(P):
    wl = synth.resnet20_workload(batch=8)
    net = P.Net(wl.ops, 8, wl.in_shape, wl.stage_end, [4, 3, 2, 1])
    xs, ys = synth.batches(wl, 12, 8)
    xs, ys = torch.from_numpy(xs).cuda(), torch.from_numpy(ys).cuda()
    losses = torch.zeros(12, device="cuda")
    st = _table(lambda t: [3, 2, 1, 0], 12, 4)
    with pytest.raises(P.PswError):   # steps 0..2 clamp their versions
        net.capture(st, wl.lr, xs, ys, losses)
    with pytest.raises(P.PswError):   # not a multiple of the period 12
        net.capture(st[:5], wl.lr, xs, ys, losses)


def test_graph_capture_rejects_dropout(P):
    """A replay would repeat the captured steps' dropout masks."""
    wl = synth.vgg16_workload(batch=2, dropout=0.3)
    net = P.Net(wl.ops, 2, wl.in_shape, wl.stage_end, [4, 3, 2, 1])
    net.load_params(synth.init_params(wl))
    xs, ys = synth.batches(wl, 12, 2)
    xs, ys = torch.from_numpy(xs).cuda(), torch.from_numpy(ys).cuda()
    losses = torch.zeros(12, device="cuda")
    st = _table(lambda t: [3, 2, 1, 0], 12, 4)
    net.pipeline_run(0, st[:3], wl.lr, xs[:3], ys[:3], losses[:3], wl.momentum)
    with pytest.raises(P.PswError) as e:
        net.capture(st, wl.lr, xs, ys, losses)
    assert e.value.code == -3


# ---- the other configurations at full size, against stored oracle runs ----
FULL_CASES = [
    ("alexnet", lambda: synth.alexnet_workload(), 20),
    ("vgg16", lambda: synth.vgg16_workload(), 40),
    ("resnet110", lambda: synth.resnet110_workload(), 3),
]


@pytest.mark.parametrize("name,factory,T", FULL_CASES, ids=[c[0] for c in FULL_CASES])
def test_full_size_against_oracle(P, name, factory, T):
    """Full-size AlexNet (b128, 20 steps), VGG-16-BN (b128, 30 stale + 10
    non-pipelined steps) and ResNet-110 (b256, bf16 products, 8 stages, 3
    steps), run as the pipelined execution, against the oracle's stored run
    (tests/golden/make_golden.py).  A trajectory check: versions exact;
    losses within the target (2e-3 fp32 / 2e-2 bf16) or 4x the oracle's own
    distance between runs on inputs one ulp apart, whichever is larger; the
    update of a seeded sample of 200,000 parameters within the target or 4x
    that spread, but never above 0.9 (a run that applied no update is at
    1.0).  VGG-16's trajectory amplifies rounding so much that the oracle
    moves 45% of its own update between the two runs; the tight bar for
    every configuration is one step from identical states
    (tests/test_gpu_onestep.py)."""
    path = os.path.join(GOLDEN, f"{name}_full_{T}steps.npz")
    if not os.path.exists(path):
        pytest.skip(f"{path} not generated (tests/golden/make_golden.py {name})")
    g = np.load(path)
    wl = factory()
    st = wl.staleness(T)
    net = P.Net(wl.ops, wl.batch, wl.in_shape, wl.stage_end, wl.ring_depth(T), bf16=wl.bf16)
    p0 = synth.init_params(wl)
    net.load_params(p0)
    xs, ys = synth.batches(wl, T)
    losses = torch.zeros(T, device="cuda")
    net.set_dropout_seed(wl.dropout_seed)
    ver = net.pipeline_run(0, st, wl.lr_table(T), torch.from_numpy(xs).cuda(), torch.from_numpy(ys).cuda(), losses,
                           wl.momentum, wl.weight_decay, wl.nesterov)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ver, g["versions"])
    flat = net.params(T).double().cpu().numpy()
    p0 = p0.astype(np.float64)
    layout, counts = synth.param_layout(wl)
    base = np.concatenate([[0], np.cumsum(counts)])
    norms = np.array([np.linalg.norm(flat[int(base[s]) + off:int(base[s]) + off + int(np.prod(shape))])
                      for _, _, shape, s, off in layout])
    samp = flat[g["index"]]
    s0 = p0[g["index"]]
    ubar = min(0.9, max(2e-2 if wl.bf16 else 1e-4, 4 * float(g["spread_update"])))
    lbar = max(2e-2 if wl.bf16 else 2e-3, 4 * float(g["spread_loss"]))
    d_upd = np.linalg.norm(samp - g["sample"]) / np.linalg.norm(g["sample"] - s0)
    d_sample = np.linalg.norm(samp - g["sample"]) / np.linalg.norm(g["sample"])
    d_loss = np.abs(losses.cpu().numpy() - g["losses"]).max() / np.abs(g["losses"]).max()
    nz = g["nonzero_init"]
    d_norm = np.max((np.abs(norms - g["norms"]) / np.maximum(g["norms"], 1e-30))[nz])
    print(f"{name}: update of the sample {d_upd:.2e} (bar {ubar:.2g}), loss {d_loss:.2e} (bar {lbar:.1e}); "
          f"sample {d_sample:.2e}, tensor norms {d_norm:.2e}; oracle spread update "
          f"{float(g['spread_update']):.2e} sample {float(g['spread_sample']):.2e} loss {float(g['spread_loss']):.2e}")
    assert np.isfinite(flat).all()
    assert d_upd <= ubar and d_loss <= lbar


def test_profile_replay_records_every_kernel(P):
    """Replay profiling (psw_net_profile_replay): every kernel of a step is
    recorded once per launch with a positive per-launch time, the same
    launches as with one event pair per launch."""
    wl = synth.resnet20_workload(batch=4)
    counts = {}
    for reps in (1, 5):
        net = P.Net(wl.ops, 4, wl.in_shape, wl.stage_end, [4, 3, 2, 1])
        net.load_params(synth.init_params(wl))
        net.profile(True)
        net.profile_replay(reps)
        x, y = synth.batch(wl, 0, 4)
        net.step(0, [3, 2, 1, 0], wl.lr, torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), wl.momentum)
        torch.cuda.synchronize()
        ks = net.profile_kernels()
        net.profile(False)
        assert all(k["ms"] > 0 for k in ks)
        counts[reps] = {k["name"]: k["launches"] for k in ks}
    assert counts[1] == counts[5]
    assert any(k.startswith("conv3x3_direct") for k in counts[5])


def test_bn_backward_folds_run(P):
    """ResNet-20 folds 13 of its 19 BN backward passes into the backward-data
    convs around them (7 without residual, 6 with an identity residual): a
    profiled step launches those folded kernels and 6 BN backward kernels of
    their own -- 5 that merge the sums of the dgrad after them, and one for
    the last BN whose output only the global average pool reads, which also
    does the pool's backward (no pool-backward, channel-sum, finalise or
    apply launches; in the forward pass its BN apply writes the pooled means,
    so no pool launch either) -- and its weight gradients as 6 grouped
    launches.  In the forward pass the 9 BNs before a block's second conv are
    applied by that conv while loading: 9 statistics-only launches and 10
    apply kernels for the 19 BNs."""
    wl = synth.resnet20_workload(batch=8)
    net = P.Net(wl.ops, 8, wl.in_shape, wl.stage_end, [4, 3, 2, 1])
    net.load_params(synth.init_params(wl))
    x, y = synth.batch(wl, 0, 8)
    net.profile(True)
    net.step(0, [3, 2, 1, 0], wl.lr, torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), wl.momentum)
    torch.cuda.synchronize()
    ks = net.profile_kernels()
    net.profile(False)
    count = lambda pred: sum(k["launches"] for k in ks if pred(k["name"]))
    assert count(lambda n: n.startswith("conv3x3_direct") and n.endswith("true, 1, 1, false>")) == 7
    assert count(lambda n: n.startswith("conv3x3_direct") and n.endswith("true, 1, 2, false>")) == 6
    assert count(lambda n: n.startswith("bn_bwd_partials_k")) == 5
    # (from the per-plane statistics its forward apply stored: one elementwise pass)
    assert count(lambda n: n.startswith("bn_bwd_gavg_stats_k")) == 1
    assert count(lambda n: n.startswith("bn_bwd_gavg_k")) == 0
    assert count(lambda n: n.startswith(("gavg_bwd_k", "chan_partials", "bn_bwd_finalize", "bn_bwd_apply"))) == 0
    # forward: that BN's apply kernel also writes the pooled means
    assert count(lambda n: n.startswith("gavg_fwd_k")) == 0
    assert count(lambda n: n.startswith("bn_stats_partials_k")) == 9
    assert count(lambda n: n.startswith("bn_apply_partials_k")) == 10
    assert [k for k in range(1, len(wl.ops) + 1) if not net.tensor_stored(k)] == [4 * b + 4 for b in range(9)]
    assert count(lambda n: n.startswith("conv3x3_wgrad")) == 6
