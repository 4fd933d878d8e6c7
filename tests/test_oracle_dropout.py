"""Dropout (App. A: VGG-16 is trained with dropout) in the oracle, pinned.

The masks come from Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC 2011), a counter-based generator, so
the backward pass of a mini-batch recomputes its forward's mask and every
side can draw the same mask from its own code.

Pins: the generator against the known-answer values published with that
paper's reference implementation (Random123) and against an independent
numpy implementation; the keep rate against its binomial law; the layer
against its definition and its adjoint; finite differences through a net
with dropout; a stale-schedule run with dropout against autograd fed the
numpy generator's masks."""
import numpy as np
import pytest

from paper_1912_12675_amd import synth
from tests import torch_ref

# (counter, key, output) of Philox4x32-10, Random123's known-answer tests
KAT = [
    ([0, 0, 0, 0], [0, 0], [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]),
    ([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2, [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]),
    ([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0],
     [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]),
]


@pytest.mark.parametrize("ctr,key,out", KAT)
def test_philox_known_answers(oracle, ctr, key, out):
    np.testing.assert_array_equal(oracle.philox4x32_10(ctr, key), np.array(out, dtype=np.uint32))
    np.testing.assert_array_equal(torch_ref.philox4x32_10(np.array([ctr]), key)[0], np.array(out, dtype=np.uint32))


def test_philox_two_implementations_agree(oracle):
    rng = np.random.default_rng(12)
    for _ in range(64):
        ctr = rng.integers(0, 2**32, 4, dtype=np.uint64)
        key = rng.integers(0, 2**32, 2, dtype=np.uint64)
        np.testing.assert_array_equal(oracle.philox4x32_10(ctr, key), torch_ref.philox4x32_10(ctr[None], key)[0])


@pytest.mark.parametrize("p", [0.1, 0.5, 0.9])
def test_dropout_layer(oracle, p):
    """y = mask * x / (1 - p) with the numpy generator's mask; the keep rate is
    within 5 sigma of 1 - p; dx = mask * dy / (1 - p) (the adjoint)."""
    k = synth.dropout_threshold(p)
    rng = np.random.default_rng(int(p * 10))
    n = 1 << 18
    x = rng.standard_normal(n)
    seed, op, step = 0x1234_5678_9ABC_DEF0, 7, (1 << 33) + 5
    y = oracle.dropout_fwd(x, k, seed, op, step)
    keep = torch_ref.dropout_mask(n, k, seed, op, step)
    scale = 16777216.0 / (16777216.0 - k)
    np.testing.assert_array_equal(y != 0, keep & (x != 0))
    np.testing.assert_allclose(y, np.where(keep, x * scale, 0.0), rtol=1e-15)
    q = 1.0 - k / 16777216.0
    assert abs(keep.mean() - q) <= 5 * np.sqrt(q * (1 - q) / n)
    dy = rng.standard_normal(n)
    dx = oracle.dropout_bwd(dy, k, seed, op, step)
    assert np.dot(y, dy) == pytest.approx(np.dot(x, dx), rel=1e-12)
    # a mask depends on the step, the op and the seed
    for args in ((seed, op, step + 1), (seed, op + 1, step), (seed + 1, op, step)):
        assert (torch_ref.dropout_mask(n, k, *args) != keep).mean() > 0.2 * min(p, 1 - p)


def _dropout_net():
    b = synth._Builder()
    t = b.add(synth.CONV, 0, 3, 8, 3, 1, 1, 0)
    t = b.add(synth.BN, t, 8, 8, flags=synth.F_RELU)
    t = b.add(synth.DROPOUT, t, 8, 8, synth.dropout_threshold(0.3))
    b.end_layer()
    t = b.add(synth.CONV, t, 8, 8, 3, 1, 1, synth.F_BIAS | synth.F_RELU)
    t = b.add(synth.MAXPOOL, t, 8, 8, 2, 2)
    b.end_layer()
    t = b.add(synth.DROPOUT, t, 8, 8, synth.dropout_threshold(0.5))
    b.add(synth.FC, t, 8 * 4 * 4, 10, flags=synth.F_BIAS)
    b.end_layer()
    return b.desc(), b.layer_end, (3, 8, 8)


def test_finite_differences_through_dropout(oracle):
    ops, le, ins = _dropout_net()
    se = [le[1], len(ops)]
    wl = synth.Workload("drop", ops, ins, 10, 3, le, se, lambda t: [0, 0], 1, [0.01, 0.01], seed=31)
    p0 = synth.init_params(wl).astype(np.float64)
    rng = np.random.default_rng(3)
    p0 += 0.05 * rng.standard_normal(p0.shape)
    x, y = synth.batch(wl, 0)
    kw = dict(dropout_seed=99, step=4)
    loss, g = oracle.loss_and_grad(ops, ins, se, p0, x, y, **kw)
    h = 1e-6
    for i in rng.choice(p0.size, 40, replace=False):
        pp, pm = p0.copy(), p0.copy()
        pp[i] += h
        pm[i] -= h
        fd = (oracle.loss_and_grad(ops, ins, se, pp, x, y, **kw)[0] -
              oracle.loss_and_grad(ops, ins, se, pm, x, y, **kw)[0]) / (2 * h)
        assert abs(fd - g[i]) <= 1e-6 * max(1e-3, abs(g[i])) + 1e-9, (i, fd, g[i])
    # another step draws other masks
    assert oracle.loss_and_grad(ops, ins, se, p0, x, y, dropout_seed=99, step=5)[0] != loss


def test_stale_training_with_dropout(oracle):
    """Two stages, staleness [2, 0], 5 steps: the oracle against the stale
    schedule in autograd (float64) whose dropout masks come from the numpy
    generator."""
    ops, le, ins = _dropout_net()
    se = [le[1], len(ops)]
    T = 5
    wl = synth.Workload("drop", ops, ins, 10, 4, le, se, lambda t: [2, 0], T, [0.02, 0.03], seed=32,
                        dropout_seed=0xDEAD_BEEF_0000_0001)
    p0 = synth.init_params(wl)
    xs, ys = synth.batches(wl, T)
    out = oracle.train(ops, ins, se, p0, xs, ys, wl.staleness(T), wl.lr, 0.9, dropout_seed=wl.dropout_seed)
    ref_p, ref_l, _ = torch_ref.train_stale(ops, se, p0, xs, ys, wl.staleness(T), wl.lr, 0.9,
                                            dropout_seed=wl.dropout_seed)
    np.testing.assert_allclose(out["losses"], ref_l, rtol=1e-10)
    np.testing.assert_allclose(out["params"], ref_p, rtol=1e-9, atol=1e-12)
    other = oracle.train(ops, ins, se, p0, xs, ys, wl.staleness(T), wl.lr, 0.9, dropout_seed=1)
    assert np.abs(other["params"] - out["params"]).max() > 1e-8
