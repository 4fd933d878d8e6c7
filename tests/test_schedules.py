"""Learning-rate policies of App. A / B and the two-partition ResNet
configurations of Table 5, and the oracle under per-step learning rates.

Pins: the step and halving policies against torch.optim.lr_scheduler
(MultiStepLR, StepLR) stepped once per mini-batch; the inverse policy at
closed-form points; Table 5's PPVs against the layer numbering; the oracle
with a per-step, per-stage rate table against the stale schedule written
with autograd (tests/torch_ref.py), with the table changing inside the run."""
import numpy as np
import pytest
import torch

from paper_1912_12675_amd import synth
from tests import torch_ref


def _torch_rates(make_sched, base, T):
    p = torch.nn.Parameter(torch.zeros(1))
    opt = torch.optim.SGD([p], lr=base)
    sched = make_sched(opt)
    out = []
    for _ in range(T):
        out.append(opt.param_groups[0]["lr"])
        opt.step()
        sched.step()
    return np.array(out)


def test_step_policy_matches_multisteplr():
    f = synth.lr_step(0.1, [7, 15], 0.1)
    ref = _torch_rates(lambda o: torch.optim.lr_scheduler.MultiStepLR(o, [7, 15], 0.1), 0.1, 25)
    np.testing.assert_allclose([f(t) for t in range(25)], ref, rtol=1e-12)


def test_halving_policy_matches_steplr():
    f = synth.lr_halving(0.1, 6)
    ref = _torch_rates(lambda o: torch.optim.lr_scheduler.StepLR(o, 6, 0.5), 0.1, 30)
    np.testing.assert_allclose([f(t) for t in range(30)], ref, rtol=1e-12)


def test_inverse_policy_closed_form():
    f = synth.lr_inverse(0.01, 1e-4, 0.75)
    assert f(0) == pytest.approx(0.01)
    assert f(10000) == pytest.approx(0.01 * 2.0 ** -0.75)       # 1 + gamma t = 2
    assert f(30000) == pytest.approx(0.01 * 4.0 ** -0.75)
    v = [f(t) for t in range(0, 30001, 1000)]
    assert all(a > b for a, b in zip(v, v[1:]))


@pytest.mark.parametrize("depth", [20, 56, 110, 224, 362])
def test_two_partition_configs(depth):
    """Table 5: one register pair after layer p, the stem and (p-1)/2 basic
    blocks in partition 1; staleness [2, 0] (K = 1 cycle schedule), [0, 0]
    after the hybrid switch; BKS_2 = partition 1 at the Table 7 rate."""
    wl = synth.resnet_two_partition_workload(depth, batch=2, n_pipelined=5, steps_per_epoch=0.1)
    p = synth.TABLE5_PPV[depth]
    assert len(wl.layer_end) - 1 == depth                     # layers 1..depth
    assert wl.stage_end == [wl.layer_end[p], len(wl.ops)]
    ops = np.asarray(wl.ops)
    convs_1 = int((ops[:wl.stage_end[0], 0] == synth.CONV).sum())
    assert convs_1 == p                                       # stem + 2 convs per block, p odd
    np.testing.assert_array_equal(wl.staleness(7), [[2, 0]] * 5 + [[0, 0]] * 2)
    lr = wl.lr_table(20)
    np.testing.assert_allclose(lr[0], [synth.TABLE7_BKS2_LR[depth], 0.1])
    np.testing.assert_allclose(lr[10], [synth.TABLE7_BKS2_LR[depth] * 0.1, 0.01])   # epoch 100 = step 10
    np.testing.assert_allclose(lr[15], [synth.TABLE7_BKS2_LR[depth] * 0.01, 0.001])  # epoch 150 = step 15


def test_oracle_per_step_rates(oracle):
    """The oracle's update takes the rate of its own step and stage: a
    two-partition ResNet-20 (batch 2) with both decays inside 6 steps and the
    hybrid switch at step 4, against autograd in float64."""
    wl = synth.resnet_two_partition_workload(20, batch=2, n_pipelined=4, steps_per_epoch=0.02)
    T = 6
    xs, ys = synth.batches(wl, T, 2)
    p0 = synth.init_params(wl)
    lr = wl.lr_table(T)
    assert len(np.unique(lr[:, 1])) == 3
    out = oracle.train(wl.ops, wl.in_shape, wl.stage_end, p0, xs, ys, wl.staleness(T), lr, wl.momentum,
                       wl.weight_decay)
    ref_p, ref_l, ref_v = torch_ref.train_stale(wl.ops, wl.stage_end, p0, xs, ys, wl.staleness(T), lr, wl.momentum,
                                                wl.weight_decay)
    np.testing.assert_array_equal(out["versions"], ref_v)
    np.testing.assert_allclose(out["losses"], ref_l, rtol=1e-10)
    np.testing.assert_allclose(out["params"], ref_p, rtol=1e-9, atol=1e-12)
    # the table matters: constant first-step rates give other parameters
    const = oracle.train(wl.ops, wl.in_shape, wl.stage_end, p0, xs, ys, wl.staleness(T), lr[0], wl.momentum,
                         wl.weight_decay)
    assert np.abs(const["params"] - out["params"]).max() > 1e-8
