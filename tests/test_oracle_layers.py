"""Pins of the oracle's per-layer maths (Sec. 2 backprop) against things other
than itself: torch.nn.functional in float64 (a different implementation),
brute-force definitional loops on tiny tensors, adjoint identities, and
library bf16 rounding."""
import itertools

import numpy as np
import pytest
import torch
import torch.nn.functional as F


CONV_CASES = [
    # N, C, H, W, K, R, stride, pad
    (2, 3, 7, 6, 4, 3, 1, 1),
    (2, 3, 7, 6, 4, 3, 2, 1),
    (1, 5, 9, 9, 3, 5, 1, 2),
    (3, 2, 8, 8, 6, 5, 1, 0),
    (2, 4, 6, 5, 2, 1, 1, 0),
    (1, 4, 11, 10, 8, 3, 2, 1),
    (2, 1, 4, 4, 3, 3, 1, 2),
]


def _t(a, grad=False):
    return torch.tensor(a, dtype=torch.float64, requires_grad=grad)


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_vs_torch(oracle, case):
    N, C, H, W, K, R, st, pad = case
    rng = np.random.default_rng(hash(case) % 2**32)
    x = rng.standard_normal((N, C, H, W))
    w = rng.standard_normal((K, C, R, R))
    b = rng.standard_normal(K)
    xt, wt, bt = _t(x, True), _t(w, True), _t(b, True)
    yt = F.conv2d(xt, wt, bt, stride=st, padding=pad)
    y = oracle.conv_fwd(x, w, b, stride=st, pad=pad)
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-12, atol=1e-12)
    dy = rng.standard_normal(yt.shape)
    yt.backward(_t(dy))
    dx = oracle.conv_bwd_data(x.shape, w, dy, stride=st, pad=pad)
    dw, db = oracle.conv_bwd_weight(x, w.shape, dy, stride=st, pad=pad, bias=True)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)


def _brute_conv(x, w, st, pad):
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    P, Q = (H + 2 * pad - R) // st + 1, (W + 2 * pad - S) // st + 1
    y = np.zeros((N, K, P, Q))
    for n, k, p, q in itertools.product(range(N), range(K), range(P), range(Q)):
        acc = 0.0
        for c, r, s in itertools.product(range(C), range(R), range(S)):
            ih, iw = p * st + r - pad, q * st + s - pad
            if 0 <= ih < H and 0 <= iw < W:
                acc += x[n, c, ih, iw] * w[k, c, r, s]
        y[n, k, p, q] = acc
    return y


@pytest.mark.parametrize("st,pad", [(1, 1), (2, 1), (1, 0), (2, 2)])
def test_conv_brute_force_and_adjoints(oracle, st, pad):
    rng = np.random.default_rng(7 + st + 3 * pad)
    x = rng.standard_normal((2, 2, 5, 4))
    w = rng.standard_normal((3, 2, 3, 3))
    y = oracle.conv_fwd(x, w, stride=st, pad=pad)
    np.testing.assert_allclose(y, _brute_conv(x, w, st, pad), rtol=1e-13, atol=1e-13)
    # adjoint identities: <conv(x;w), dy> = <x, bwd_data(dy;w)> = <w, bwd_weight(x,dy)>
    dy = rng.standard_normal(y.shape)
    dx = oracle.conv_bwd_data(x.shape, w, dy, stride=st, pad=pad)
    dw = oracle.conv_bwd_weight(x, w.shape, dy, stride=st, pad=pad)
    lhs = float((y * dy).sum())
    assert abs(lhs - float((x * dx).sum())) < 1e-11 * max(1.0, abs(lhs))
    assert abs(lhs - float((w * dw).sum())) < 1e-11 * max(1.0, abs(lhs))


def test_conv_bwd_data_accumulates(oracle):
    rng = np.random.default_rng(3)
    x = rng.standard_normal((1, 2, 5, 5))
    w = rng.standard_normal((2, 2, 3, 3))
    dy = rng.standard_normal((1, 2, 5, 5))
    base = oracle.conv_bwd_data(x.shape, w, dy, 1, 1)
    # call the raw routine twice on one buffer: result doubles
    import ctypes
    dx = np.zeros(x.shape)
    L = oracle.lib()
    P = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    for _ in range(2):
        L.orc_conv_bwd_data(1, 2, 5, 5, 2, 3, 3, 1, 1, P(np.ascontiguousarray(w)), P(np.ascontiguousarray(dy)), P(dx), 0)
    np.testing.assert_allclose(dx, 2 * base, rtol=1e-14)


@pytest.mark.parametrize("residual", [None, "identity", "optionA"])
@pytest.mark.parametrize("relu", [False, True])
def test_bn_vs_torch(oracle, residual, relu):
    rng = np.random.default_rng(11 + (residual is not None) + 2 * relu)
    N, C, H, W = 3, 4, 5, 6
    y = rng.standard_normal((N, C, H, W)) * 2.0 + 0.7
    g = rng.uniform(0.5, 1.5, C)
    be = rng.standard_normal(C)
    res = None
    if residual == "identity":
        res = rng.standard_normal((N, C, H, W))
    elif residual == "optionA":
        res = rng.standard_normal((N, C // 2, 2 * H, 2 * W))
    yt, gt, bt = _t(y, True), _t(g, True), _t(be, True)
    rm_t, rv_t = torch.zeros(C, dtype=torch.float64), torch.ones(C, dtype=torch.float64)
    zt = F.batch_norm(yt, rm_t, rv_t, gt, bt, training=True, momentum=0.1, eps=1e-5)
    rt = None
    if res is not None:
        rt = _t(res, True)
        if residual == "identity":
            zt = zt + rt
        else:
            lo = (C - C // 2) // 2
            zt = zt + F.pad(rt[:, :, ::2, ::2], (0, 0, 0, 0, lo, C - C // 2 - lo))
    if relu:
        zt = F.relu(zt)
    rm, rv = np.zeros(C), np.ones(C)
    z, mean, invstd = oracle.bn_fwd(y, g, be, res=res, relu=relu, run_mean=rm, run_var=rv)
    np.testing.assert_allclose(z, zt.detach().numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(rm, rm_t.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(rv, rv_t.numpy(), rtol=1e-12, atol=1e-14)
    dz = rng.standard_normal(z.shape)
    zt.backward(_t(dz))
    dy, dg, db, dres = oracle.bn_bwd(dz, z, y, g, mean, invstd, relu=relu,
                                     res_shape=None if res is None else res.shape)
    np.testing.assert_allclose(dy, yt.grad.numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-11, atol=1e-11)
    if res is not None:
        np.testing.assert_allclose(dres, rt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_bn_normalises(oracle):
    """Closed form: with gamma=1, beta=0 the output has mean 0 and biased
    variance var/(var+eps) per channel."""
    rng = np.random.default_rng(5)
    y = rng.standard_normal((4, 3, 5, 5)) * np.array([1.0, 3.0, 0.2])[None, :, None, None] + 5.0
    z, mean, invstd = oracle.bn_fwd(y, np.ones(3), np.zeros(3))
    var = y.var(axis=(0, 2, 3))
    np.testing.assert_allclose(z.mean(axis=(0, 2, 3)), 0.0, atol=1e-13)
    np.testing.assert_allclose(z.var(axis=(0, 2, 3)), var / (var + 1e-5), rtol=1e-12)
    np.testing.assert_allclose(mean, y.mean(axis=(0, 2, 3)), rtol=1e-13)


@pytest.mark.parametrize("shape,k,st", [((2, 3, 8, 8), 2, 2), ((1, 2, 7, 9), 2, 2), ((2, 2, 9, 9), 3, 3)])
def test_maxpool_vs_torch(oracle, shape, k, st):
    rng = np.random.default_rng(sum(shape))
    x = rng.standard_normal(shape)
    xt = _t(x, True)
    yt, it = F.max_pool2d(xt, k, st, return_indices=True)
    y, am = oracle.maxpool_fwd(x, k, st)
    np.testing.assert_array_equal(y, yt.detach().numpy())
    np.testing.assert_array_equal(am, it.numpy())
    dy = rng.standard_normal(y.shape)
    yt.backward(_t(dy))
    dx = oracle.maxpool_bwd(x.shape, k, st, dy, am)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=0, atol=0)


def test_maxpool_first_max_on_ties(oracle):
    x = np.zeros((1, 1, 2, 2))
    y, am = oracle.maxpool_fwd(x, 2, 2)
    assert am[0, 0, 0, 0] == 0
    x = np.array([[[[1.0, 3.0], [3.0, 2.0]]]])
    y, am = oracle.maxpool_fwd(x, 2, 2)
    assert am[0, 0, 0, 0] == 1 and y[0, 0, 0, 0] == 3.0


def test_gavgpool(oracle):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 4, 8, 8))
    y = oracle.gavgpool_fwd(x)
    np.testing.assert_allclose(y, x.mean(axis=(2, 3)), rtol=1e-14)
    dy = rng.standard_normal((3, 4))
    dx = oracle.gavgpool_bwd(x.shape, dy)
    np.testing.assert_allclose(dx, np.broadcast_to(dy[:, :, None, None] / 64, x.shape), rtol=1e-14)


def test_fc_vs_torch(oracle):
    rng = np.random.default_rng(4)
    x, w, b = rng.standard_normal((5, 7)), rng.standard_normal((3, 7)), rng.standard_normal(3)
    xt, wt, bt = _t(x, True), _t(w, True), _t(b, True)
    yt = F.linear(xt, wt, bt)
    np.testing.assert_allclose(oracle.fc_fwd(x, w, b), yt.detach().numpy(), rtol=1e-13)
    dy = rng.standard_normal((5, 3))
    yt.backward(_t(dy))
    dx, dw, db = oracle.fc_bwd(x, w, dy)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-13)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-13)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-13)


def test_softmax_xent_vs_torch(oracle):
    rng = np.random.default_rng(6)
    z = rng.standard_normal((9, 10)) * 4
    lab = rng.integers(0, 10, 9).astype(np.int32)
    zt = _t(z, True)
    lt = F.cross_entropy(zt, torch.tensor(lab, dtype=torch.long))
    lt.backward()
    loss, dz = oracle.softmax_xent(z, lab)
    assert abs(loss - float(lt)) < 1e-13
    np.testing.assert_allclose(dz, zt.grad.numpy(), rtol=1e-12, atol=1e-15)


def test_softmax_xent_uniform_logits(oracle):
    """Closed form: equal logits give loss log(C)."""
    loss, dz = oracle.softmax_xent(np.zeros((4, 10)), np.arange(4, dtype=np.int32))
    assert abs(loss - np.log(10)) < 1e-14
    np.testing.assert_allclose(dz.sum(axis=1), 0.0, atol=1e-16)


@pytest.mark.parametrize("nesterov,wd", [(False, 0.0), (False, 1e-4), (True, 5e-4)])
def test_sgd_vs_torch(oracle, nesterov, wd):
    rng = np.random.default_rng(8)
    w0 = rng.standard_normal(50)
    p = _t(w0, True)
    opt = torch.optim.SGD([p], lr=0.05, momentum=0.9, weight_decay=wd, nesterov=nesterov)
    w, v = w0.copy(), np.zeros(50)
    for step in range(4):
        g = rng.standard_normal(50)
        p.grad = _t(g)
        opt.step()
        w, v = oracle.sgd(w, v, g, 0.05, 0.9, wd, nesterov)
    np.testing.assert_allclose(w, p.detach().numpy(), rtol=1e-14, atol=1e-15)


def test_bf16_rounding_matches_library(oracle):
    """The bf16 switch rounds each product operand to bfloat16 (nearest
    even): conv on the switch == fp64 conv on torch-rounded operands."""
    rng = np.random.default_rng(9)
    x = rng.standard_normal((2, 3, 6, 6)).astype(np.float32).astype(np.float64)
    w = rng.standard_normal((4, 3, 3, 3)).astype(np.float32).astype(np.float64)
    xr = torch.tensor(x).float().bfloat16().double().numpy()
    wr = torch.tensor(w).float().bfloat16().double().numpy()
    y = oracle.conv_fwd(x, w, stride=1, pad=1, bf16=True)
    np.testing.assert_allclose(y, oracle.conv_fwd(xr, wr, stride=1, pad=1), rtol=1e-14, atol=1e-14)
    assert np.abs(y - oracle.conv_fwd(x, w, stride=1, pad=1)).max() > 1e-4
    a = rng.standard_normal((5, 8)).astype(np.float32).astype(np.float64)
    b = rng.standard_normal((3, 8)).astype(np.float32).astype(np.float64)
    ar = torch.tensor(a).float().bfloat16().double().numpy()
    br = torch.tensor(b).float().bfloat16().double().numpy()
    np.testing.assert_allclose(oracle.fc_fwd(a, b, bf16=True), ar @ br.T, rtol=1e-14, atol=1e-14)
    # ties to even on exact halfway cases
    h = np.array([[1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8]])
    one = np.ones((1, 2))
    out = oracle.fc_fwd(h, np.eye(2), bf16=True)
    np.testing.assert_array_equal(out, [[1.0, 1.0 + 2 * 2.0 ** -7]])
    assert one.shape == (1, 2)
