"""Thin ctypes binding of libpsw (include/psw.h).

Every function here only marshals arguments: tensors become device pointers,
sizes become C ints, and a non-zero status becomes a PswError carrying
psw_last_error().  All computation happens in the HIP kernels of libpsw.so.
PyTorch provides device memory and the current stream.

The library must be built first (``python -m paper_1912_12675_amd.build``);
loading fails loudly when it is missing.  torch is imported before the
library so that both share one HIP runtime.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpsw.so")

PSW_OK = 0
PSW_ERR = {-1: "NULL", -2: "SHAPE", -3: "UNSUPPORTED", -4: "STALENESS", -5: "STEP_ORDER", -6: "WORKSPACE",
           -7: "HIP", -8: "STATE"}
PSW_FP32, PSW_BF16 = 0, 1
PSW_POOL_MAX, PSW_POOL_GAVG = 0, 1

_I, _I64, _F, _P, _SZ = ctypes.c_int, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t


class PswError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"psw error {code} ({PSW_ERR.get(code, '?')}): {msg}")
        self.code = code


class psw_layer(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("kind", "in0", "in1", "cin", "cout", "k", "stride", "pad", "flags")]


class psw_launch(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("what", ctypes.c_int32), ("stage", ctypes.c_int32),
                ("version", ctypes.c_int64)]


class psw_kernel_span(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 96), ("kind", ctypes.c_int32), ("stream", ctypes.c_int32),
                ("start_us", ctypes.c_double), ("end_us", ctypes.c_double)]


class psw_kernel_stat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 192), ("kind", ctypes.c_int32), ("launches", ctypes.c_int64),
                ("ms", ctypes.c_double), ("flops", ctypes.c_double), ("bytes", ctypes.c_double)]


# symbol -> (restype, argtypes); the full public surface of include/psw.h
SIGNATURES = {
    "psw_last_error": (ctypes.c_char_p, []),
    "psw_version": (ctypes.c_char_p, []),
    "psw_conv_fwd": (_I, [_I] * 9 + [_P, _P, _P, _I, _P, _I, _P]),
    "psw_conv_bwd_data": (_I, [_I] * 9 + [_P, _P, _P, _I, _I, _P]),
    "psw_conv_bwd_weight_ws_bytes": (_SZ, [_I] * 10),
    "psw_conv_bwd_weight": (_I, [_I] * 9 + [_P, _P, _P, _P, _I, _P, _SZ, _P]),
    "psw_conv_bwd_weight_noalloc": (_I, [_I] * 9 + [_P, _P, _P, _P, _I, _P]),
    "psw_bn_ws_bytes": (_SZ, [_I] * 4),
    "psw_bn_relu_fwd": (_I, [_I] * 4 + [_P, _P, _P, _P, _I, _I, _I, _I, _F, _F, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "psw_bn_relu_bwd": (_I, [_I] * 4 + [_P] * 6 + [_I, _P, _P, _P, _P, _I, _I, _I, _I, _P, _SZ, _P]),
    "psw_pool_fwd": (_I, [_I] * 7 + [_P, _P, _P, _P]),
    "psw_pool_bwd": (_I, [_I] * 7 + [_P, _P, _P, _I, _P]),
    "psw_fc_fwd": (_I, [_I] * 3 + [_P, _P, _P, _I, _P, _I, _P]),
    "psw_fc_bwd_ws_bytes": (_SZ, [_I] * 3),
    "psw_fc_bwd": (_I, [_I] * 3 + [_P, _P, _P, _P, _I, _P, _P, _I, _P, _SZ, _P]),
    "psw_relu_mask": (_I, [_I64, _P, _P, _P]),
    "psw_softmax_xent": (_I, [_I, _I, _P, _P, _P, _P, _P]),
    "psw_sgd_momentum_step": (_I, [_I64, _P, _P, _P, _P, _F, _F, _F, _I, _P]),
    "psw_dropout": (_I, [_I64, _P, _P, _I, _I, ctypes.c_uint64, ctypes.c_int32, _I64, _P]),
    "psw_net_set_dropout_seed": (_I, [_P, ctypes.c_uint64]),
    "psw_net_create": (_I, [ctypes.POINTER(psw_layer), _I, _I, _I, _I, _I, _P, _I, _P, _I,
                            ctypes.POINTER(ctypes.c_void_p)]),
    "psw_net_destroy": (None, [_P]),
    "psw_net_sizes": (_I, [_P, _P, _P, _P, _P, _P]),
    "psw_net_bind": (_I, [_P, _P, _P, _P, _P, _P, _P, _SZ]),
    "psw_stage_step": (_I, [_P, _I64, _P, _P, _F, _F, _I, _P, _P, _P, _P, _P]),
    "psw_net_set_step": (_I, [_P, _I64]),
    "psw_net_set_weight_stashing": (_I, [_P, _I]),
    "psw_net_slot": (_I, [_P, _I, _I64, ctypes.POINTER(ctypes.c_void_p)]),
    "psw_net_param_offset": (_I, [_P, _I, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int64),
                                  ctypes.POINTER(ctypes.c_int64)]),
    "psw_net_tensor": (_I, [_P, _I, _I, ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(ctypes.c_int64)]),
    "psw_net_tensor_stored": (_I, [_P, _I, ctypes.POINTER(ctypes.c_int)]),
    "psw_net_bn_saved": (_I, [_P, _I] + [ctypes.POINTER(ctypes.c_void_p)] * 3),
    "psw_net_set_bn_on_load": (_I, [_P, _I]),
    "psw_net_plan": (_I, [_P, _I64, _P, ctypes.POINTER(psw_launch), _I, ctypes.POINTER(ctypes.c_int)]),
    "psw_net_profile": (_I, [_P, _I]),
    "psw_net_profile_read": (_I, [_P, _I, _P, _P]),
    "psw_net_profile_kernels": (_I, [_P, _I, _P, _P]),
    "psw_net_profile_only": (_I, [_P, _I, ctypes.c_char_p]),
    "psw_net_profile_replay": (_I, [_P, _I]),
    "psw_net_profile_timeline": (_I, [_P, _I, _P, _P]),
    "psw_net_pipeline_bytes": (_I, [_P, _P]),
    "psw_net_bind_pipeline": (_I, [_P, _P, _SZ]),
    "psw_pipeline_run": (_I, [_P, _I64, _I, _P, _P, _F, _F, _I, _P, _P, _I, _P, _P, _P]),
    "psw_pipeline_capture": (_I, [_P, _I, _P, _P, _F, _F, _I, _P, _P, _I, _P, _P]),
    "psw_graph_launch": (_I, [_P, _P]),
    "psw_graph_destroy": (_I, [_P]),
}

PROF_KINDS = ["conv_fwd", "conv_bwd_data", "conv_bwd_weight", "bn_fwd", "bn_bwd", "pool", "fc", "loss", "sgd",
              "other"]

_lib = None


def lib():
    """Load libpsw.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_1912_12675_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(rc: int):
    if rc != PSW_OK:
        raise PswError(rc, lib().psw_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, torch.Tensor):
        if not t.is_cuda:
            raise ValueError("libpsw takes device tensors")
        if not t.is_contiguous():
            raise ValueError("libpsw takes contiguous tensors")
        if t.dtype not in (torch.float32, torch.int32, torch.uint8):
            raise TypeError(f"libpsw takes float32 / int32 buffers (workspaces uint8), got {t.dtype}")
        return t.data_ptr()
    raise TypeError(type(t))


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _prec(bf16):
    return PSW_BF16 if bf16 else PSW_FP32


# ------------------------------------------------------------ per layer ----
def psw_conv_fwd(x, w, y, stride=1, pad=0, bias=None, relu=False, bf16=False, stream=None):
    n, c, h, wd = x.shape
    k, _, r, s = w.shape
    _check(lib().psw_conv_fwd(n, c, h, wd, k, r, s, stride, pad, _ptr(x), _ptr(w), _ptr(bias), int(relu), _ptr(y),
                              _prec(bf16), _stream(stream)))


def psw_conv_bwd_data(x_shape, w, dy, dx, stride=1, pad=0, accumulate=False, bf16=False, stream=None):
    n, c, h, wd = x_shape
    k, _, r, s = w.shape
    _check(lib().psw_conv_bwd_data(n, c, h, wd, k, r, s, stride, pad, _ptr(w), _ptr(dy), _ptr(dx), int(accumulate),
                                   _prec(bf16), _stream(stream)))


def psw_conv_bwd_weight_ws_bytes(x_shape, w_shape, stride=1, pad=0, bf16=False):
    n, c, h, wd = x_shape
    k, _, r, s = w_shape
    return int(lib().psw_conv_bwd_weight_ws_bytes(n, c, h, wd, k, r, s, stride, pad, _prec(bf16)))


def psw_conv_bwd_weight(x, dy, dw, stride=1, pad=0, dbias=None, bf16=False, ws=None, stream=None):
    n, c, h, wd = x.shape
    k, _, r, s = dw.shape
    if ws is None:
        nb = psw_conv_bwd_weight_ws_bytes(x.shape, dw.shape, stride, pad, bf16)
        ws = torch.empty(max(nb, 1), dtype=torch.uint8, device=x.device)
    _check(lib().psw_conv_bwd_weight(n, c, h, wd, k, r, s, stride, pad, _ptr(x), _ptr(dy), _ptr(dw), _ptr(dbias),
                                     _prec(bf16), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def psw_conv_bwd_weight_noalloc(x, dy, dw, stride=1, pad=0, dbias=None, bf16=False, stream=None):
    """psw_conv_bwd_weight without a workspace (the library's static scratch)."""
    N, C, H, W = x.shape
    K, _, R, S = dw.shape
    _check(lib().psw_conv_bwd_weight_noalloc(N, C, H, W, K, R, S, stride, pad, _ptr(x), _ptr(dy), _ptr(dw),
                                             _ptr(dbias), _prec(bf16), _stream(stream)))


def psw_bn_ws_bytes(shape):
    return int(lib().psw_bn_ws_bytes(*[int(v) for v in shape]))


def _ws(nbytes, device):
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def psw_bn_relu_fwd(y, gamma, beta, z, save_mean, save_invstd, res=None, relu=False, eps=1e-5, momentum=0.1,
                    run_mean=None, run_var=None, ws=None, stream=None):
    n, c, h, w = y.shape
    rc, rh, rw = (0, 0, 0) if res is None else tuple(res.shape[1:])
    ws = _ws(psw_bn_ws_bytes(y.shape), y.device) if ws is None else ws
    _check(lib().psw_bn_relu_fwd(n, c, h, w, _ptr(y), _ptr(gamma), _ptr(beta), _ptr(res), rc, rh, rw, int(relu),
                                 eps, momentum, _ptr(z), _ptr(save_mean), _ptr(save_invstd), _ptr(run_mean),
                                 _ptr(run_var), _ptr(ws), ws.numel(), _stream(stream)))


def psw_bn_relu_bwd(dz, z, y, gamma, save_mean, save_invstd, dy, dgamma, dbeta, dres=None, relu=False,
                    res_accumulate=False, ws=None, stream=None):
    n, c, h, w = y.shape
    rc, rh, rw = (0, 0, 0) if dres is None else tuple(dres.shape[1:])
    ws = _ws(psw_bn_ws_bytes(y.shape), y.device) if ws is None else ws
    _check(lib().psw_bn_relu_bwd(n, c, h, w, _ptr(dz), _ptr(z), _ptr(y), _ptr(gamma), _ptr(save_mean),
                                 _ptr(save_invstd), int(relu), _ptr(dy), _ptr(dgamma), _ptr(dbeta), _ptr(dres), rc, rh,
                                 rw, int(res_accumulate), _ptr(ws), ws.numel(), _stream(stream)))


def psw_pool_fwd(kind, x, y, k=2, stride=2, argmax=None, stream=None):
    n, c, h, w = x.shape
    _check(lib().psw_pool_fwd(kind, n, c, h, w, k, stride, _ptr(x), _ptr(y), _ptr(argmax), _stream(stream)))


def psw_pool_bwd(kind, x_shape, dy, dx, k=2, stride=2, argmax=None, accumulate=False, stream=None):
    n, c, h, w = x_shape
    _check(lib().psw_pool_bwd(kind, n, c, h, w, k, stride, _ptr(dy), _ptr(argmax), _ptr(dx), int(accumulate),
                              _stream(stream)))


def psw_fc_fwd(x, w, y, b=None, relu=False, bf16=False, stream=None):
    n, fin = x.shape
    out = w.shape[0]
    _check(lib().psw_fc_fwd(n, fin, out, _ptr(x), _ptr(w), _ptr(b), int(relu), _ptr(y), _prec(bf16),
                            _stream(stream)))


def psw_fc_bwd_ws_bytes(n, fin, out):
    return int(lib().psw_fc_bwd_ws_bytes(n, fin, out))


def psw_fc_bwd(x, w, dy, dw, dx=None, db=None, dx_accumulate=False, bf16=False, ws=None, stream=None):
    n, fin = x.shape
    out = w.shape[0]
    ws = _ws(psw_fc_bwd_ws_bytes(n, fin, out), x.device) if ws is None else ws
    _check(lib().psw_fc_bwd(n, fin, out, _ptr(x), _ptr(w), _ptr(dy), _ptr(dx), int(dx_accumulate), _ptr(dw), _ptr(db),
                            _prec(bf16), _ptr(ws), ws.numel(), _stream(stream)))


def psw_relu_mask(z, g, stream=None):
    _check(lib().psw_relu_mask(z.numel(), _ptr(z), _ptr(g), _stream(stream)))


def psw_softmax_xent(logits, labels, loss, dlogits, stream=None):
    n, classes = logits.shape
    _check(lib().psw_softmax_xent(n, classes, _ptr(logits), _ptr(labels), _ptr(loss), _ptr(dlogits),
                                  _stream(stream)))


def psw_sgd_momentum_step(w_in, w_out, v, g, lr, mom=0.9, wd=0.0, nesterov=False, stream=None):
    _check(lib().psw_sgd_momentum_step(w_in.numel(), _ptr(w_in), _ptr(w_out), _ptr(v), _ptr(g), lr, mom, wd,
                                       int(nesterov), _stream(stream)))


def psw_dropout(x, y, p24, seed, op, t, accumulate=False, stream=None):
    """y (+)= keep * x * 2^24 / (2^24 - p24), the Philox mask of (seed, op, t)."""
    _check(lib().psw_dropout(x.numel(), _ptr(x), _ptr(y), int(accumulate), int(p24), int(seed), int(op), int(t),
                             _stream(stream)))


# ------------------------------------------------------------- networks ----
def _layers(ops):
    ops = np.ascontiguousarray(ops, dtype=np.int32).reshape(-1, 9)
    arr = (psw_layer * len(ops))()
    for i, o in enumerate(ops):
        arr[i] = psw_layer(*[int(v) for v in o])
    return arr


class Graph:
    """A captured pipelined run (psw_pipeline_capture); keeps the captured tensors alive."""

    def __init__(self, handle, keep):
        self.handle, self._keep = handle, keep

    def launch(self, stream=None):
        _check(lib().psw_graph_launch(self.handle, _stream(stream)))

    def __del__(self):
        h = getattr(self, "handle", None)
        if h and _lib is not None:
            _lib.psw_graph_destroy(h)
            self.handle = None


class Net:
    """A network bound to torch-allocated device buffers.

    Wraps psw_net_create / psw_net_sizes / psw_net_bind / psw_stage_step.
    ``ring`` holds every stage's weight-version slots; ``load_params`` writes
    W^(0) (the packed stage parameters, stages concatenated) into slot 0.
    """

    def __init__(self, ops, batch, in_shape, stage_end, ring_depth, bf16=False, device="cuda", step_sets=3):
        L = lib()
        if step_sets not in (2, 3):
            raise ValueError(f"step_sets must be 2 or 3, got {step_sets}")
        self.step_sets = step_sets  # step sets a pipelined run rotates (psw_net_bind_pipeline)
        self.ops = np.ascontiguousarray(ops, dtype=np.int32).reshape(-1, 9)
        self.S = len(stage_end)
        self._layers = _layers(self.ops)
        se = np.ascontiguousarray(stage_end, dtype=np.int32)
        rd = np.ascontiguousarray(ring_depth, dtype=np.int32)
        h = ctypes.c_void_p()
        _check(L.psw_net_create(self._layers, len(self.ops), batch, *[int(v) for v in in_shape], se.ctypes.data,
                                self.S, rd.ctypes.data, _prec(bf16), ctypes.byref(h)))
        self.handle = h.value
        self.ring_depth = [int(v) for v in rd]
        sp = np.zeros(self.S, dtype=np.int64)
        rf, npar, nbn, ab = (ctypes.c_int64() for _ in range(4))
        _check(L.psw_net_sizes(self.handle, sp.ctypes.data, ctypes.byref(rf), ctypes.byref(npar), ctypes.byref(nbn),
                               ctypes.byref(ab)))
        self.ring_floats, self.arena_bytes = rf.value, ab.value
        self.stage_params = [int(v) for v in sp]
        self.n_params = npar.value
        dev = torch.device(device)
        self.ring = torch.zeros(max(rf.value, 1), dtype=torch.float32, device=dev)
        self.momentum = torch.zeros(max(npar.value, 1), dtype=torch.float32, device=dev)
        self.grad = torch.zeros(max(npar.value, 1), dtype=torch.float32, device=dev)
        self.run_mean = torch.zeros(max(nbn.value, 1), dtype=torch.float32, device=dev)
        self.run_var = torch.ones(max(nbn.value, 1), dtype=torch.float32, device=dev)
        self.arena = torch.empty(max(ab.value, 256), dtype=torch.uint8, device=dev)
        self.loss = torch.zeros(1, dtype=torch.float32, device=dev)
        self.bn_channels = nbn.value
        _check(L.psw_net_bind(self.handle, _ptr(self.ring), _ptr(self.momentum), _ptr(self.grad),
                              _ptr(self.run_mean), _ptr(self.run_var), _ptr(self.arena), self.arena.numel()))
        self.device = dev

    def __del__(self):
        h = getattr(self, "handle", None)
        if h and _lib is not None:
            _lib.psw_net_destroy(h)
            self.handle = None

    def _slot_index(self, stage, version):
        p = ctypes.c_void_p()
        _check(lib().psw_net_slot(self.handle, stage, version, ctypes.byref(p)))
        off = (p.value - self.ring.data_ptr()) // 4
        return off

    def slot(self, stage, version):
        """View of stage `stage`'s weight version `version` inside the ring."""
        off = self._slot_index(stage, version)
        return self.ring[off:off + self.stage_params[stage]]

    def load_params(self, flat):
        """Write W^(0) (stages concatenated) into slot 0 of every stage."""
        flat = torch.as_tensor(flat, dtype=torch.float32)
        o = 0
        for s in range(self.S):
            n = self.stage_params[s]
            self.slot(s, 0).copy_(flat[o:o + n].to(self.device))
            o += n

    def params(self, version):
        """All stages' parameters at `version` (concatenated, float32 on host)."""
        return torch.cat([self.slot(s, version).detach().cpu() for s in range(self.S)])

    def tensor(self, tensor, grad=False):
        """View of tensor `tensor` (op tensor-1's output) of the last
        psw_stage_step, or of its gradient (psw_net_tensor)."""
        p, n = ctypes.c_void_p(), ctypes.c_int64()
        _check(lib().psw_net_tensor(self.handle, int(tensor), int(bool(grad)), ctypes.byref(p), ctypes.byref(n)))
        off = p.value - self.arena.data_ptr()
        return self.arena[off:off + 4 * n.value].view(torch.float32)

    def tensor_stored(self, tensor):
        """False for the output of a BN applied by its consumer conv while
        loading (psw_net_tensor_stored): its psw_net_tensor view holds no value."""
        st = ctypes.c_int()
        _check(lib().psw_net_tensor_stored(self.handle, int(tensor), ctypes.byref(st)))
        return bool(st.value)

    def bn_saved(self, op):
        """Views of BN op `op`'s saved mean [c], invstd [c] and scale_shift [2c] of the last
        psw_stage_step (psw_net_bn_saved)."""
        ptrs = [ctypes.c_void_p() for _ in range(3)]
        _check(lib().psw_net_bn_saved(self.handle, int(op), *[ctypes.byref(q) for q in ptrs]))
        c = int(self.ops[op][3])
        out = []
        for q, n in zip(ptrs, (c, c, 2 * c)):
            off = q.value - self.arena.data_ptr()
            out.append(self.arena[off:off + 4 * n].view(torch.float32))
        return tuple(out)

    def set_bn_on_load(self, on=True):
        """BNs applied by their one consumer conv while loading (default) or stored by their own kernel."""
        _check(lib().psw_net_set_bn_on_load(self.handle, int(bool(on))))

    def set_step(self, t):
        _check(lib().psw_net_set_step(self.handle, int(t)))

    def set_dropout_seed(self, seed):
        _check(lib().psw_net_set_dropout_seed(self.handle, int(seed)))

    def set_weight_stashing(self, on=True):
        """Backward data gradients with the forward's version (comparison scheme)."""
        _check(lib().psw_net_set_weight_stashing(self.handle, int(bool(on))))

    def step(self, t, staleness, lr, x, labels, mom=0.9, wd=0.0, nesterov=False, stream=None):
        st = np.ascontiguousarray(staleness, dtype=np.int32)
        lrs = np.ascontiguousarray(np.broadcast_to(np.asarray(lr, dtype=np.float32), (self.S,)))
        ver = np.zeros(self.S, dtype=np.int32)
        _check(lib().psw_stage_step(self.handle, int(t), st.ctypes.data, lrs.ctypes.data, mom, wd, int(nesterov),
                                    _ptr(x), _ptr(labels), _ptr(self.loss), ver.ctypes.data, _stream(stream)))
        return ver

    def pipeline_run(self, t0, staleness, lr, xs, labels, losses, mom=0.9, wd=0.0, nesterov=False, stream=None):
        """Steps t0 .. t0+n-1 as a pipeline (psw_pipeline_run): staleness [n, S] and lr ([n, S] or [S] or scalar)
        host arrays; xs [n_batches, batch, ...] and labels [n_batches, batch] device tensors (step t0+i uses batch
        i mod n_batches); losses: device float32 tensor of n entries.  Returns the versions [n, S]."""
        self._ensure_pipeline_set()
        st = np.ascontiguousarray(staleness, dtype=np.int32).reshape(-1, self.S)
        n = st.shape[0]
        lrs = np.ascontiguousarray(np.broadcast_to(np.asarray(lr, dtype=np.float32), (n, self.S)))
        assert losses.numel() >= n and xs.shape[0] == labels.shape[0]
        ver = np.zeros((n, self.S), dtype=np.int32)
        _check(lib().psw_pipeline_run(self.handle, int(t0), n, st.ctypes.data, lrs.ctypes.data, mom, wd,
                                      int(nesterov), _ptr(xs), _ptr(labels), int(xs.shape[0]), _ptr(losses),
                                      ver.ctypes.data, _stream(stream)))
        return ver

    def _ensure_pipeline_set(self):
        if getattr(self, "step2", None) is None:
            nb = ctypes.c_int64()
            _check(lib().psw_net_pipeline_bytes(self.handle, ctypes.byref(nb)))
            extra = self.step_sets - 1  # sets beside the arena
            self.step2 = torch.empty(max(extra * nb.value, 256), dtype=torch.uint8, device=self.device)
            _check(lib().psw_net_bind_pipeline(self.handle, _ptr(self.step2), self.step2.numel()))

    def device_bytes(self):
        """Device memory the net holds: the ring, momentum, gradient and running
        statistics vectors, the arena (one step set and the shared workspaces)
        and, once a pipelined run has bound them, the extra step sets."""
        held = [self.ring, self.momentum, self.grad, self.run_mean, self.run_var, self.arena]
        if getattr(self, "step2", None) is not None:
            held.append(self.step2)
        return sum(t.numel() * t.element_size() for t in held)

    def capture(self, staleness, lr, xs, labels, losses, mom=0.9, wd=0.0, nesterov=False):
        """Capture the next n pipelined steps into a graph (psw_pipeline_capture); returns a Graph whose
        launch() runs the next n steps each time.  The tensors passed must outlive the graph."""
        self._ensure_pipeline_set()
        st = np.ascontiguousarray(staleness, dtype=np.int32).reshape(-1, self.S)
        n = st.shape[0]
        lrs = np.ascontiguousarray(np.broadcast_to(np.asarray(lr, dtype=np.float32), (n, self.S)))
        g = ctypes.c_void_p()
        _check(lib().psw_pipeline_capture(self.handle, n, st.ctypes.data, lrs.ctypes.data, mom, wd, int(nesterov),
                                          _ptr(xs), _ptr(labels), int(xs.shape[0]), _ptr(losses), ctypes.byref(g)))
        return Graph(g.value, (self, xs, labels, losses))

    def profile(self, enable=True, only=None):
        """Enable / disable HIP-event timing of the kernels launched by step() (all of them, or only the
        kernel named `only`); clears the records."""
        if only:
            _check(lib().psw_net_profile_only(self.handle, int(enable), only.encode()))
        else:
            _check(lib().psw_net_profile(self.handle, int(enable)))

    def profile_read(self):
        """{kind: (milliseconds, kernel launches)} summed over the records."""
        ms = np.zeros(len(PROF_KINDS), dtype=np.float64)
        cnt = np.zeros(len(PROF_KINDS), dtype=np.int64)
        _check(lib().psw_net_profile_read(self.handle, len(PROF_KINDS), ms.ctypes.data, cnt.ctypes.data))
        return {k: (float(ms[i]), int(cnt[i])) for i, k in enumerate(PROF_KINDS)}

    def profile_replay(self, reps):
        """Time every recorded launch in isolation as reps back-to-back launches (reps 1: one event pair
        per launch); the replayed run's numbers are not the schedule's."""
        _check(lib().psw_net_profile_replay(self.handle, int(reps)))

    def profile_timeline(self, cap=1 << 20):
        """[(name, kind, stream, start_us, end_us)] per recorded launch, in issue order."""
        n = ctypes.c_int()
        _check(lib().psw_net_profile_timeline(self.handle, 0, None, ctypes.byref(n)))
        buf = (psw_kernel_span * max(1, min(n.value, cap)))()
        _check(lib().psw_net_profile_timeline(self.handle, min(n.value, cap), buf, ctypes.byref(n)))
        return [(buf[i].name.decode(), PROF_KINDS[buf[i].kind] if 0 <= buf[i].kind < len(PROF_KINDS) else "other",
                 int(buf[i].stream), float(buf[i].start_us), float(buf[i].end_us)) for i in range(min(n.value, cap))]

    def profile_kernels(self, cap=256):
        """[{name, kind, launches, ms, flops, bytes}] per distinct kernel, in decreasing total time."""
        buf = (psw_kernel_stat * cap)()
        n = ctypes.c_int()
        _check(lib().psw_net_profile_kernels(self.handle, cap, buf, ctypes.byref(n)))
        return [dict(name=buf[i].name.decode(), kind=PROF_KINDS[buf[i].kind] if 0 <= buf[i].kind < len(PROF_KINDS)
                     else "other", launches=int(buf[i].launches), ms=float(buf[i].ms), flops=float(buf[i].flops),
                     bytes=float(buf[i].bytes)) for i in range(min(n.value, cap))]

    def plan(self, t, staleness, cap=4096):
        st = np.ascontiguousarray(staleness, dtype=np.int32)
        buf = (psw_launch * cap)()
        n = ctypes.c_int()
        _check(lib().psw_net_plan(self.handle, int(t), st.ctypes.data, buf, cap, ctypes.byref(n)))
        return [(buf[i].op, buf[i].what, buf[i].stage, buf[i].version) for i in range(min(n.value, cap))]


def net_plan_only(ops, batch, in_shape, stage_end, ring_depth, t, staleness, bf16=False, cap=4096, stash=False):
    """psw_net_create + psw_net_plan without binding any memory (host only)."""
    L = lib()
    layers = _layers(ops)
    se = np.ascontiguousarray(stage_end, dtype=np.int32)
    rd = np.ascontiguousarray(ring_depth, dtype=np.int32)
    h = ctypes.c_void_p()
    _check(L.psw_net_create(layers, len(layers), batch, *[int(v) for v in in_shape], se.ctypes.data, len(se),
                            rd.ctypes.data, _prec(bf16), ctypes.byref(h)))
    try:
        st = np.ascontiguousarray(staleness, dtype=np.int32)
        buf = (psw_launch * cap)()
        n = ctypes.c_int()
        _check(L.psw_net_set_weight_stashing(h.value, int(bool(stash))))
        _check(L.psw_net_plan(h.value, int(t), st.ctypes.data, buf, cap, ctypes.byref(n)))
        return [(buf[i].op, buf[i].what, buf[i].stage, buf[i].version) for i in range(min(n.value, cap))]
    finally:
        L.psw_net_destroy(h.value)
