"""ctypes binding of the CPU oracle (test infrastructure only).

The oracle is plain C in ``mtx_oracle.c``; this module only marshals numpy arrays.  It takes the
network as (C, H, W) plus a list of layer tuples (kind, out, k, stride, pad, groups, relu) with
kind 0 = fully connected, 1 = convolution, 2 = max-pool, 3 = batch normalisation, 4 = residual
addition of the output of layer k, 5 = residual addition of layer k's output through a 1x1
projection of the given stride, so it needs nothing from the GPU library.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

from . import build as _build

EHINT = -6


class _Layer(C.Structure):
    _fields_ = [(n, C.c_int) for n in ("kind", "out", "k", "stride", "pad", "groups", "relu")]


_lib = None


def lib():
    global _lib
    if _lib is None:
        path = _build.LIB
        if (not os.path.exists(path) or
                os.path.getmtime(path) < os.path.getmtime(_build.SRC)):
            _build.build()
        _lib = C.CDLL(path)
        _lib.orc_round_bf16.restype = C.c_float
        _lib.orc_round_bf16.argtypes = [C.c_float]
        _lib.orc_splitmix64_first.restype = C.c_uint64
        _lib.orc_splitmix64_first.argtypes = [C.c_uint64]
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _layers(layers: Sequence[Sequence[int]]):
    arr = (_Layer * len(layers))()
    for i, t in enumerate(layers):
        for name, val in zip(("kind", "out", "k", "stride", "pad", "groups", "relu"), t):
            setattr(arr[i], name, int(val))
    return arr


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def splitmix64_first(key: int) -> int:
    """First output of a SplitMix64 generator whose state is `key` (the oracle's init RNG)."""
    return int(lib().orc_splitmix64_first(C.c_uint64(key)))


def num_threads() -> int:
    return int(lib().orc_num_threads())


def round_bf16(x: np.ndarray) -> np.ndarray:
    f = lib().orc_round_bf16
    flat = np.asarray(x, dtype=np.float32).ravel()
    return np.array([f(float(t)) for t in flat], dtype=np.float32).reshape(np.shape(x))


def param_count(in_shape, layers) -> int:
    n = C.c_long()
    rc = lib().orc_param_count(*[C.c_int(v) for v in in_shape], C.c_int(len(layers)),
                               _layers(layers), C.byref(n))
    if rc:
        raise ValueError(f"oracle rejected the network (rc={rc})")
    return n.value


def geometry(in_shape, layers):
    """Per-layer (input shape, output shape, w_off, w_len, b_off, b_len) from the oracle's plan,
    computed in Python from the same definitions for convenience of the tests."""
    c, h, w = in_shape
    off = 0
    out = []
    for (kind, o, k, s, p, g, relu) in layers:
        if kind == 1:
            oc, oh, ow = o, (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
            wl, bl = o * (c // g) * k * k, o
        elif kind == 0:
            oc, oh, ow = o, 1, 1
            wl, bl = o * c * h * w, o
        elif kind == 3:  # batch normalisation: gamma, beta per channel
            oc, oh, ow = c, h, w
            wl, bl = c, c
        elif kind == 4:  # residual addition of layer k's output
            oc, oh, ow = c, h, w
            wl, bl = 0, 0
        elif kind == 5:  # addition through a 1x1 projection of layer k's output
            oc, oh, ow = c, h, w
            wl, bl = o * out[k]["out_shape"][0], o
        else:
            oc, oh, ow = c, (h - k) // s + 1, (w - k) // s + 1
            wl, bl = 0, 0
        out.append(dict(kind=kind, relu=relu, k=k, in_shape=(c, h, w), out_shape=(oc, oh, ow),
                        w_off=off, w_len=wl, b_off=off + wl, b_len=bl))
        off += wl + bl
        c, h, w = oc, oh, ow
    return out


def init_glorot(in_shape, layers, seed: int) -> np.ndarray:
    P = param_count(in_shape, layers)
    w = np.empty(P, dtype=np.float32)
    rc = lib().orc_init_glorot(*[C.c_int(v) for v in in_shape], C.c_int(len(layers)),
                               _layers(layers), C.c_uint64(seed), _p(w))
    if rc:
        raise ValueError(f"orc_init_glorot rc={rc}")
    return w


# ---- single layers in double precision ------------------------------------------------------

def conv_fwd(x, w, b, stride, pad, groups):
    x, w = _f64(x), _f64(w)
    N, Cc, H, W = x.shape
    OC, _, K, _ = w.shape
    OH, OW = (H + 2 * pad - K) // stride + 1, (W + 2 * pad - K) // stride + 1
    y = np.empty((N, OC, OH, OW))
    lib().orc_conv_fwd(*[C.c_int(v) for v in (N, Cc, H, W, OC, K, stride, pad, groups)],
                       _p(x), _p(w), _p(None if b is None else _f64(b)), _p(y))
    return y


def conv_bwd(x, w, dy, stride, pad, groups, need_dx=True):
    x, w, dy = _f64(x), _f64(w), _f64(dy)
    N, Cc, H, W = x.shape
    OC, _, K, _ = w.shape
    dx = np.empty_like(x) if need_dx else None
    dw = np.empty_like(w)
    db = np.empty(OC)
    lib().orc_conv_bwd(*[C.c_int(v) for v in (N, Cc, H, W, OC, K, stride, pad, groups)],
                       _p(x), _p(w), _p(dy), _p(dx), _p(dw), _p(db))
    return dx, dw, db


def fc_fwd(x, w, b):
    x, w = _f64(x), _f64(w)
    N, IN = x.shape
    OUT = w.shape[0]
    y = np.empty((N, OUT))
    lib().orc_fc_fwd(C.c_int(N), C.c_int(IN), C.c_int(OUT), _p(x), _p(w),
                     _p(None if b is None else _f64(b)), _p(y))
    return y


def fc_bwd(x, w, dy, need_dx=True):
    x, w, dy = _f64(x), _f64(w), _f64(dy)
    N, IN = x.shape
    OUT = w.shape[0]
    dx = np.empty_like(x) if need_dx else None
    dw = np.empty_like(w)
    db = np.empty(OUT)
    lib().orc_fc_bwd(C.c_int(N), C.c_int(IN), C.c_int(OUT), _p(x), _p(w), _p(dy), _p(dx),
                     _p(dw), _p(db))
    return dx, dw, db


def maxpool_fwd(x, k, s):
    x = _f64(x)
    N, Cc, H, W = x.shape
    OH, OW = (H - k) // s + 1, (W - k) // s + 1
    y = np.empty((N, Cc, OH, OW))
    am = np.empty((N, Cc, OH, OW), dtype=np.int32)
    lib().orc_maxpool_fwd(*[C.c_int(v) for v in (N, Cc, H, W, k, s)], _p(x), _p(y), _p(am))
    return y, am


def maxpool_bwd(x_shape, k, s, argmax, dy):
    N, Cc, H, W = x_shape
    dx = np.empty(x_shape)
    am = np.ascontiguousarray(argmax, dtype=np.int32)
    lib().orc_maxpool_bwd(*[C.c_int(v) for v in (N, Cc, H, W, k, s)], _p(am), _p(_f64(dy)),
                          _p(dx))
    return dx


def softmax_xent(z, labels, scale):
    z = _f64(z)
    N, NC = z.shape
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    loss = np.empty(N)
    dz = np.empty_like(z)
    lib().orc_softmax_xent(C.c_int(N), C.c_int(NC), _p(z), _p(lab), C.c_double(scale),
                           _p(loss), _p(dz))
    return loss, dz


# ---- the training step ------------------------------------------------------------------------

@dataclass
class StepResult:
    loss: float
    shard_loss: np.ndarray
    grads: Optional[np.ndarray]  # [R, P]
    gavg: np.ndarray
    w_new: np.ndarray
    v_new: Optional[np.ndarray]
    acts: Optional[np.ndarray]
    pool_argmax: Optional[np.ndarray]
    relu_mask: Optional[np.ndarray]


class HintRejected(RuntimeError):
    pass


def decision_sizes(in_shape, layers, batch):
    """Sizes of the concatenated activation / pool-decision / ReLU-decision arrays."""
    geo = geometry(in_shape, layers)
    act = sum(int(np.prod(g["out_shape"])) * batch for g in geo)
    pool = sum(int(np.prod(g["out_shape"])) * batch for g in geo if g["kind"] == 2)
    relu = sum(int(np.prod(g["out_shape"])) * batch for g in geo if g["relu"])
    return act, pool, relu


PREC = {"f32": 0, "bf16": 1, "exact": 2}

# Default window of a decision hint, relative to the scale of the layer's values: the per-tensor
# tolerance of the comparisons of stored outputs in each precision mode.
HINT_REL = {"f32": 1e-4, "bf16": 2e-2, "exact": 1e-4}


def train_step(in_shape, layers, R, x, labels, w, v, lr, mu, prec="f32", want_grads=True,
               want_acts=False, want_decisions=False, pool_hint=None, relu_hint=None,
               hint_rel=None):
    """One step of the oracle (see orc_train_step).  hint_rel is the window of a decision hint
    relative to the layer's scale; by default HINT_REL[prec]."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    w = np.ascontiguousarray(w, dtype=np.float32)
    v = None if v is None else np.ascontiguousarray(v, dtype=np.float32)
    B = x.shape[0]
    if B % R:
        raise ValueError("batch must split into R equal shards")
    Nb = B // R
    P = param_count(in_shape, layers)
    n_act, n_pool, n_relu = decision_sizes(in_shape, layers, B)
    loss = C.c_double()
    shard_loss = np.empty(R, dtype=np.float32)
    grads = np.empty((R, P), dtype=np.float32) if want_grads else None
    gavg = np.empty(P, dtype=np.float32)
    w_new = np.empty(P, dtype=np.float32)
    v_new = np.empty(P, dtype=np.float32)
    acts = np.empty(n_act, dtype=np.float32) if want_acts else None
    pam = np.empty(n_pool, dtype=np.int32) if want_decisions else None
    rmask = np.empty(n_relu, dtype=np.int8) if want_decisions else None
    ph = None if pool_hint is None else np.ascontiguousarray(pool_hint, dtype=np.int32)
    rh = None if relu_hint is None else np.ascontiguousarray(relu_hint, dtype=np.int8)
    if ph is not None and ph.size != n_pool:
        raise ValueError("pool_hint has the wrong size")
    if rh is not None and rh.size != n_relu:
        raise ValueError("relu_hint has the wrong size")
    rc = lib().orc_train_step(
        *[C.c_int(t) for t in in_shape], C.c_int(len(layers)), _layers(layers), C.c_int(R),
        C.c_int(Nb), C.c_int(PREC[prec]), _p(x), _p(labels), _p(w), _p(v),
        C.c_float(lr), C.c_float(mu), _p(ph), _p(rh),
        C.c_double(HINT_REL[prec] if hint_rel is None else hint_rel), C.byref(loss),
        _p(shard_loss), _p(grads),
        _p(gavg), _p(w_new), _p(v_new), _p(acts), _p(pam), _p(rmask))
    if rc == EHINT:
        raise HintRejected("a decision hint lies outside the oracle's window for it")
    if rc:
        raise RuntimeError(f"orc_train_step rc={rc}")
    return StepResult(loss.value, shard_loss, grads, gavg, w_new, v_new if v is not None else None,
                      acts, pam, rmask)


def average_update(grads, w, v, lr, mu, n=None):
    """Average of the rows of grads (R x ld, first n columns) fused with the momentum update.
    Returns (gavg, w_new, v_new)."""
    grads = np.ascontiguousarray(grads, dtype=np.float32)
    R, ld = grads.shape
    n = ld if n is None else n
    w2 = np.array(w, dtype=np.float32, copy=True)
    v2 = None if v is None else np.array(v, dtype=np.float32, copy=True)
    gavg = np.empty(n, dtype=np.float32)
    rc = lib().orc_average_update(_p(grads), C.c_int(R), C.c_long(n), C.c_long(ld), _p(w2),
                                  _p(v2), C.c_float(lr), C.c_float(mu), _p(gavg))
    if rc:
        raise RuntimeError(f"orc_average_update rc={rc}")
    return gavg, w2, v2


def average_adam(grads, w, m, v, lr, b1, b2, eps, step, n=None):
    """Average of the rows of grads (R x ld, first n columns) followed by one Adam step number
    `step` (>= 1).  Returns (gavg, w_new, m_new, v_new)."""
    grads = np.ascontiguousarray(grads, dtype=np.float32)
    R, ld = grads.shape
    n = ld if n is None else n
    w2, m2, v2 = (np.array(a, dtype=np.float32, copy=True) for a in (w, m, v))
    gavg = np.empty(n, dtype=np.float32)
    rc = lib().orc_average_adam(_p(grads), C.c_int(R), C.c_long(n), C.c_long(ld), _p(w2),
                                _p(m2), _p(v2), C.c_float(lr), C.c_float(b1), C.c_float(b2),
                                C.c_float(eps), C.c_long(step), _p(gavg))
    if rc:
        raise RuntimeError(f"orc_average_adam rc={rc}")
    return gavg, w2, m2, v2


def average_adagrad(grads, w, acc, lr, eps, n=None):
    """Average of the rows of grads followed by one AdaGrad step.  Returns
    (gavg, w_new, acc_new)."""
    grads = np.ascontiguousarray(grads, dtype=np.float32)
    R, ld = grads.shape
    n = ld if n is None else n
    w2, a2 = (np.array(a, dtype=np.float32, copy=True) for a in (w, acc))
    gavg = np.empty(n, dtype=np.float32)
    rc = lib().orc_average_adagrad(_p(grads), C.c_int(R), C.c_long(n), C.c_long(ld), _p(w2),
                                   _p(a2), C.c_float(lr), C.c_float(eps), _p(gavg))
    if rc:
        raise RuntimeError(f"orc_average_adagrad rc={rc}")
    return gavg, w2, a2
