"""ctypes wrapper around the plain C oracle (``psw_oracle.c``).

TEST INFRASTRUCTURE ONLY: the oracle is the slow, obviously-correct CPU
reference for pipelined training with stale weights (Zhang & Abdelrahman,
arXiv 1912.12675).  Only the test suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this module.  It shares no code
with the GPU library.

Every array is float64 except inputs (float32, as drawn by the harness),
labels and versions (int32).  Layouts: NCHW activations, KCRS conv weights,
[out][in] FC weights.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "psw_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (-O2, OpenMP).  Portable x86-64 code: no
    -march=native, so the same build runs on any host."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-Wno-unknown-pragmas", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = ctypes.CDLL(_LIB)
        _declare(_lib)
    return _lib


_d = ctypes.POINTER(ctypes.c_double)
_f = ctypes.POINTER(ctypes.c_float)
_i32 = ctypes.POINTER(ctypes.c_int32)
_i64 = ctypes.POINTER(ctypes.c_int64)
_I = ctypes.c_int
_i64v = ctypes.c_int64
_D = ctypes.c_double


def _declare(L):
    L.orc_num_threads.restype = _I
    L.orc_set_num_threads.argtypes = [_I]
    L.orc_conv_fwd.argtypes = [_I] * 9 + [_d, _d, _d, _d, _I]
    L.orc_conv_bwd_data.argtypes = [_I] * 9 + [_d, _d, _d, _I]
    L.orc_conv_bwd_weight.argtypes = [_I] * 9 + [_d, _d, _d, _d, _I]
    L.orc_bn_fwd.argtypes = [_I] * 4 + [_d, _d, _d, _d, _I, _I, _I, _I, _D, _d, _d, _d, _d, _d, _D]
    L.orc_bn_bwd.argtypes = [_I] * 4 + [_d, _d, _d, _d, _d, _d, _I, _d, _d, _d, _d, _I, _I, _I]
    L.orc_maxpool_fwd.argtypes = [_I] * 6 + [_d, _d, _i32]
    L.orc_maxpool_bwd.argtypes = [_I] * 6 + [_d, _i32, _d]
    L.orc_gavgpool_fwd.argtypes = [_I] * 4 + [_d, _d]
    L.orc_gavgpool_bwd.argtypes = [_I] * 4 + [_d, _d]
    L.orc_fc_fwd.argtypes = [_I] * 3 + [_d, _d, _d, _d, _I]
    L.orc_fc_bwd.argtypes = [_I] * 3 + [_d, _d, _d, _d, _d, _d, _I]
    L.orc_softmax_xent.argtypes = [_I, _I, _d, _i32, _d]
    L.orc_softmax_xent.restype = _D
    L.orc_sgd.argtypes = [ctypes.c_int64, _d, _d, _d, _d, _D, _D, _D, _I]
    L.orc_param_counts.argtypes = [_I, _i32, _I, _I, _I, _I, _I, _i32, _i64]
    L.orc_param_counts.restype = _I
    L.orc_shapes.argtypes = [_I, _i32, _I, _I, _I, _I, _I, _i32, _i32]
    L.orc_shapes.restype = _I
    L.orc_train_from.argtypes = [_I, _i32, _I, _I, _I, _I, _I, _i32, _i64v, _I, _d, _d, _I, _I, _f, _i32, _i32, _d,
                                 _D, _D, _I, _D, _D, _I, _I, _I, _d, _d, _d, _d, _d, _d, _i32, ctypes.c_uint64]
    L.orc_loss_and_grad.argtypes = [_I, _i32, _I, _I, _I, _I, _I, _i32, _d, _f, _i32, _D, _I,
                                    _d, _d, _d, ctypes.c_uint64, _i64v]
    L.orc_loss_and_grad.restype = _I
    L.orc_train.argtypes = [_I, _i32, _I, _I, _I, _I, _I, _i32, _d, _I, _f, _i32, _i32, _d,
                            _D, _D, _I, _D, _D, _I, _I, _d, _d, _d, _d, _d, _i32, ctypes.c_uint64]
    _u32 = ctypes.POINTER(ctypes.c_uint32)
    L.orc_philox4x32_10.argtypes = [_u32, _u32, _u32]
    L.orc_philox4x32_10.restype = None
    L.orc_dropout_fwd.argtypes = [_i64v, _d, _d, _I, ctypes.c_uint64, _I, _i64v]
    L.orc_dropout_fwd.restype = None
    L.orc_dropout_bwd.argtypes = [_i64v, _d, _d, _I, ctypes.c_uint64, _I, _i64v]
    L.orc_dropout_bwd.restype = None
    L.orc_train.restype = _I


def _p(a, kind):
    if a is None:
        return None
    return a.ctypes.data_as(kind)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def set_threads(n: int) -> None:
    lib().orc_set_num_threads(int(n))


def num_threads() -> int:
    return int(lib().orc_num_threads())


# ---------------------------------------------------------------- layers ----
def conv_out(h, k, stride, pad):
    return (h + 2 * pad - k) // stride + 1


def conv_fwd(x, w, b=None, stride=1, pad=0, bf16=False):
    x, w = _f64(x), _f64(w)
    N, C, H, W = x.shape
    K, C2, R, S = w.shape
    assert C2 == C
    P, Q = conv_out(H, R, stride, pad), conv_out(W, S, stride, pad)
    y = np.zeros((N, K, P, Q))
    bb = None if b is None else _f64(b)
    lib().orc_conv_fwd(N, C, H, W, K, R, S, stride, pad, _p(x, _d), _p(w, _d), _p(bb, _d),
                       _p(y, _d), int(bf16))
    return y


def conv_bwd_data(x_shape, w, dy, stride=1, pad=0, bf16=False):
    w, dy = _f64(w), _f64(dy)
    N, C, H, W = x_shape
    K, _, R, S = w.shape
    dx = np.zeros((N, C, H, W))
    lib().orc_conv_bwd_data(N, C, H, W, K, R, S, stride, pad, _p(w, _d), _p(dy, _d), _p(dx, _d),
                            int(bf16))
    return dx


def conv_bwd_weight(x, w_shape, dy, stride=1, pad=0, bias=False, bf16=False):
    x, dy = _f64(x), _f64(dy)
    N, C, H, W = x.shape
    K, _, R, S = w_shape
    dw = np.zeros((K, C, R, S))
    db = np.zeros(K) if bias else None
    lib().orc_conv_bwd_weight(N, C, H, W, K, R, S, stride, pad, _p(x, _d), _p(dy, _d), _p(dw, _d),
                              _p(db, _d), int(bf16))
    return (dw, db) if bias else dw


def bn_fwd(y, gamma, beta, res=None, relu=False, eps=1e-5, run_mean=None, run_var=None, momentum=0.1):
    y, gamma, beta = _f64(y), _f64(gamma), _f64(beta)
    N, C, H, W = y.shape
    z = np.zeros_like(y)
    mean, invstd = np.zeros(C), np.zeros(C)
    r = None if res is None else _f64(res)
    Cr, Hr, Wr = (0, 0, 0) if r is None else r.shape[1:]
    lib().orc_bn_fwd(N, C, H, W, _p(y, _d), _p(gamma, _d), _p(beta, _d), _p(r, _d), Cr, Hr, Wr,
                     int(relu), eps, _p(z, _d), _p(mean, _d), _p(invstd, _d), _p(run_mean, _d),
                     _p(run_var, _d), momentum)
    return z, mean, invstd


def bn_bwd(dz, z, y, gamma, mean, invstd, relu=False, res_shape=None):
    dz, z, y, gamma, mean, invstd = map(_f64, (dz, z, y, gamma, mean, invstd))
    N, C, H, W = y.shape
    dy = np.zeros_like(y)
    dg, db = np.zeros(C), np.zeros(C)
    dres = None if res_shape is None else np.zeros(res_shape)
    Cr, Hr, Wr = (0, 0, 0) if res_shape is None else res_shape[1:]
    lib().orc_bn_bwd(N, C, H, W, _p(dz, _d), _p(z, _d), _p(y, _d), _p(gamma, _d), _p(mean, _d),
                     _p(invstd, _d), int(relu), _p(dy, _d), _p(dg, _d), _p(db, _d), _p(dres, _d),
                     Cr, Hr, Wr)
    return dy, dg, db, dres


def maxpool_fwd(x, k, stride):
    x = _f64(x)
    N, C, H, W = x.shape
    P, Q = (H - k) // stride + 1, (W - k) // stride + 1
    y = np.zeros((N, C, P, Q))
    am = np.zeros((N, C, P, Q), dtype=np.int32)
    lib().orc_maxpool_fwd(N, C, H, W, k, stride, _p(x, _d), _p(y, _d), _p(am, _i32))
    return y, am


def maxpool_bwd(x_shape, k, stride, dy, argmax):
    dy = _f64(dy)
    argmax = np.ascontiguousarray(argmax, dtype=np.int32)
    N, C, H, W = x_shape
    dx = np.zeros((N, C, H, W))
    lib().orc_maxpool_bwd(N, C, H, W, k, stride, _p(dy, _d), _p(argmax, _i32), _p(dx, _d))
    return dx


def gavgpool_fwd(x):
    x = _f64(x)
    N, C, H, W = x.shape
    y = np.zeros((N, C))
    lib().orc_gavgpool_fwd(N, C, H, W, _p(x, _d), _p(y, _d))
    return y


def gavgpool_bwd(x_shape, dy):
    dy = _f64(dy)
    N, C, H, W = x_shape
    dx = np.zeros((N, C, H, W))
    lib().orc_gavgpool_bwd(N, C, H, W, _p(dy, _d), _p(dx, _d))
    return dx


def fc_fwd(x, w, b=None, bf16=False):
    x, w = _f64(x), _f64(w)
    N, In = x.shape
    Out = w.shape[0]
    y = np.zeros((N, Out))
    bb = None if b is None else _f64(b)
    lib().orc_fc_fwd(N, In, Out, _p(x, _d), _p(w, _d), _p(bb, _d), _p(y, _d), int(bf16))
    return y


def fc_bwd(x, w, dy, bias=True, bf16=False):
    x, w, dy = _f64(x), _f64(w), _f64(dy)
    N, In = x.shape
    Out = w.shape[0]
    dx = np.zeros((N, In))
    dw = np.zeros((Out, In))
    db = np.zeros(Out) if bias else None
    lib().orc_fc_bwd(N, In, Out, _p(x, _d), _p(w, _d), _p(dy, _d), _p(dx, _d), _p(dw, _d),
                     _p(db, _d), int(bf16))
    return dx, dw, db


def softmax_xent(z, labels):
    z = _f64(z)
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    N, Cls = z.shape
    dz = np.zeros_like(z)
    loss = lib().orc_softmax_xent(N, Cls, _p(z, _d), _p(labels, _i32), _p(dz, _d))
    return float(loss), dz


def sgd(w, v, g, lr, mom=0.9, wd=0.0, nesterov=False):
    """Returns (w_new, v_new); inputs are not modified."""
    w = _f64(w).copy()
    v = _f64(v).copy()
    g = _f64(g)
    out = np.empty_like(w)
    lib().orc_sgd(w.size, _p(w, _d), _p(out, _d), _p(v, _d), _p(g, _d), lr, mom, wd, int(nesterov))
    return out, v


# --------------------------------------------------------------- networks ---
def _desc(ops):
    return np.ascontiguousarray(ops, dtype=np.int32).reshape(-1, 9)


def param_counts(ops, in_shape, batch, stage_end):
    ops = _desc(ops)
    se = np.ascontiguousarray(stage_end, dtype=np.int32)
    out = np.zeros(len(se), dtype=np.int64)
    rc = lib().orc_param_counts(len(ops), _p(ops, _i32), batch, *in_shape, len(se), _p(se, _i32),
                                _p(out, _i64))
    if rc != 0:
        raise ValueError(f"oracle rejected the network description (code {rc})")
    return out


def shapes(ops, in_shape, batch, stage_end):
    ops = _desc(ops)
    se = np.ascontiguousarray(stage_end, dtype=np.int32)
    out = np.zeros((len(ops) + 1, 4), dtype=np.int32)
    rc = lib().orc_shapes(len(ops), _p(ops, _i32), batch, *in_shape, len(se), _p(se, _i32),
                          _p(out, _i32))
    if rc != 0:
        raise ValueError(f"oracle rejected the network description (code {rc})")
    return out


def philox4x32_10(counter, key):
    """Philox4x32-10 of a 4-word counter under a 2-word key (uint32 words)."""
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    u32 = ctypes.POINTER(ctypes.c_uint32)
    lib().orc_philox4x32_10(c.ctypes.data_as(u32), k.ctypes.data_as(u32), out.ctypes.data_as(u32))
    return out


def dropout_fwd(x, p24, seed, op, step):
    x = _f64(x)
    y = np.zeros_like(x)
    lib().orc_dropout_fwd(x.size, _p(x, _d), _p(y, _d), int(p24), int(seed), int(op), int(step))
    return y


def dropout_bwd(dy, p24, seed, op, step):
    dy = _f64(dy)
    dx = np.zeros_like(dy)
    lib().orc_dropout_bwd(dy.size, _p(dy, _d), _p(dx, _d), int(p24), int(seed), int(op), int(step))
    return dx


def loss_and_grad(ops, in_shape, stage_end, params, x, labels, bn_eps=1e-5, bf16=False,
                  want_acts=False, dropout_seed=0, step=0):
    ops = _desc(ops)
    se = np.ascontiguousarray(stage_end, dtype=np.int32)
    params = _f64(params)
    x = np.ascontiguousarray(x, dtype=np.float32)
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    N = x.shape[0]
    grads = np.zeros_like(params)
    acts = None
    if want_acts:
        shp = shapes(ops, in_shape, N, stage_end)
        acts = np.zeros(int(np.prod(shp, axis=1).sum()))
    loss = ctypes.c_double(0.0)
    rc = lib().orc_loss_and_grad(len(ops), _p(ops, _i32), N, *in_shape, len(se), _p(se, _i32),
                                 _p(params, _d), _p(x, _f), _p(labels, _i32), bn_eps, int(bf16),
                                 ctypes.byref(loss), _p(grads, _d), _p(acts, _d), int(dropout_seed), int(step))
    if rc != 0:
        raise ValueError(f"oracle rejected the network description (code {rc})")
    if want_acts:
        return loss.value, grads, acts
    return loss.value, grads


def train(ops, in_shape, stage_end, params0, xs, labels, staleness, lr, mom=0.9, wd=0.0,
          nesterov=False, bn_eps=1e-5, bn_mom=0.1, bf16=False, stash=False, dropout_seed=0):
    """Run T steps of the stale-weight schedule.  xs: [T, N, C, H, W] float32;
    labels [T, N]; staleness [T, S]; lr: scalar, [S] or [T, S] (per step and
    stage).  stash=True: the backward pass takes its
    data gradients with the forward's weight version (weight stashing, the
    scheme Sec. 6.7 contrasts with) instead of the current one.  Returns a dict
    with params, momentum, run_mean, run_var, losses and versions."""
    ops = _desc(ops)
    se = np.ascontiguousarray(stage_end, dtype=np.int32)
    S = len(se)
    xs = np.ascontiguousarray(xs, dtype=np.float32)
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    T, N = xs.shape[0], xs.shape[1]
    stal = np.ascontiguousarray(staleness, dtype=np.int32).reshape(T, S)
    lr = np.asarray(lr, dtype=np.float64)
    lr = np.ascontiguousarray(np.broadcast_to(lr if lr.ndim == 2 else np.broadcast_to(lr, (S,)), (T, S)))
    params0 = _f64(params0)
    out = np.zeros_like(params0)
    momb = np.zeros_like(params0)
    n_bn = int(sum(o[4] for o in ops if o[0] == 2))
    rm, rv = np.zeros(max(n_bn, 1)), np.zeros(max(n_bn, 1))
    losses = np.zeros(T)
    versions = np.zeros((T, S), dtype=np.int32)
    rc = lib().orc_train(len(ops), _p(ops, _i32), N, *in_shape, S, _p(se, _i32), _p(params0, _d), T,
                         _p(xs, _f), _p(labels, _i32), _p(stal, _i32), _p(lr, _d), mom, wd,
                         int(nesterov), bn_eps, bn_mom, int(bf16), int(stash), _p(out, _d), _p(momb, _d),
                         _p(rm, _d), _p(rv, _d), _p(losses, _d), _p(versions, _i32), int(dropout_seed))
    if rc != 0:
        raise ValueError(f"oracle rejected the run (code {rc})")
    return dict(params=out, momentum=momb, run_mean=rm[:n_bn], run_var=rv[:n_bn], losses=losses,
                versions=versions)


def train_from(ops, in_shape, stage_end, t0, hist0, mom0, xs, labels, staleness, lr, mom=0.9, wd=0.0,
               nesterov=False, bn_eps=1e-5, bn_mom=0.1, bf16=False, stash=False, dropout_seed=0,
               run_mean=None, run_var=None, out_depth=1):
    """Resume the stale-weight schedule from a checkpoint at step t0 and run
    len(xs) steps (t0 .. t0+T-1; batch i is step t0+i's).

    hist0: [S][depth] list of per-stage packed parameter vectors, versions
    t0-depth+1 .. t0 (entries of negative versions may be None); mom0: the
    concatenated momentum at t0 (None: zero); run_mean / run_var: the
    running statistics at t0 (None: mean 0, var 1).  staleness [T, S]; lr
    scalar, [S] or [T, S].  Returns a dict with `history` ([S][out_depth]
    vectors W_s^(t0+T-out_depth+1) .. W_s^(t0+T), None below version 0),
    `params` (W^(t0+T) concatenated), `momentum`, `grad` (the last step's
    gradient), `run_mean`, `run_var`, `losses` and `versions`."""
    ops = _desc(ops)
    se = np.ascontiguousarray(stage_end, dtype=np.int32)
    S = len(se)
    counts = param_counts(ops, in_shape, 1, stage_end)
    depth = len(hist0[0])
    assert all(len(h) == depth for h in hist0), "every stage needs the same number of versions"
    packed = np.zeros(depth * int(sum(counts)))
    o = 0
    for s in range(S):
        for k in range(depth):
            v = hist0[s][k]
            if v is not None:
                packed[o + k * counts[s]:o + (k + 1) * counts[s]] = np.asarray(v, dtype=np.float64)
        o += depth * counts[s]
    xs = np.ascontiguousarray(xs, dtype=np.float32)
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    T = xs.shape[0]
    stal = np.ascontiguousarray(staleness, dtype=np.int32).reshape(T, S)
    lr = np.asarray(lr, dtype=np.float64)
    lr = np.ascontiguousarray(np.broadcast_to(lr if lr.ndim == 2 else np.broadcast_to(lr, (S,)), (T, S)))
    n = int(sum(counts))
    m0 = None if mom0 is None else _f64(mom0)
    n_bn = int(sum(o[4] for o in ops if o[0] == 2))
    rm, rv = np.zeros(max(n_bn, 1)), np.ones(max(n_bn, 1))
    bn_in = run_mean is not None
    if bn_in:
        rm[:n_bn] = run_mean
        rv[:n_bn] = run_var
    hist_out = np.zeros(out_depth * n)
    momb, grad = np.zeros(n), np.zeros(n)
    losses = np.zeros(T)
    versions = np.zeros((T, S), dtype=np.int32)
    rc = lib().orc_train_from(len(ops), _p(ops, _i32), xs.shape[1], *in_shape, S, _p(se, _i32), int(t0), depth,
                              _p(packed, _d), _p(m0, _d), int(bn_in), T, _p(xs, _f), _p(labels, _i32),
                              _p(stal, _i32), _p(lr, _d), mom, wd, int(nesterov), bn_eps, bn_mom, int(bf16),
                              int(stash), out_depth, _p(hist_out, _d), _p(momb, _d), _p(grad, _d), _p(rm, _d),
                              _p(rv, _d), _p(losses, _d), _p(versions, _i32), int(dropout_seed))
    if rc != 0:
        raise ValueError(f"oracle rejected the run (code {rc})")
    history, o = [], 0
    for s in range(S):
        row = []
        for k in range(out_depth):
            v = t0 + T - out_depth + 1 + k
            row.append(hist_out[o + k * counts[s]:o + (k + 1) * counts[s]].copy() if v >= 0 else None)
        history.append(row)
        o += out_depth * counts[s]
    params = np.concatenate([h[-1] for h in history])
    return dict(history=history, params=params, momentum=momb, grad=grad, run_mean=rm[:n_bn], run_var=rv[:n_bn],
                losses=losses, versions=versions)
