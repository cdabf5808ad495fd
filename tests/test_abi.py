"""The C ABI library on the host: it loads, exports every entry point include/mtx.h declares,
sizes the paper's networks like the oracle does, and rejects invalid arguments before touching
a GPU (these calls need no device)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from oracle import oracle as orc
from paper_1704_04560_amd import mtx
from paper_1704_04560_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "mtx.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mtx_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = _declared()
    assert len(names) >= 11
    lib = C.CDLL(mtx.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(mtx.EXPORTS)


@pytest.mark.parametrize("name", list(wl.WORKLOADS))
def test_sizes_match_oracle(name):
    w = wl.WORKLOADS[name]
    layers = wl.layer_tuples(w.net)
    d = mtx.make_desc(w.net.in_shape, layers, w.net.dtype)
    P, ld, ws = mtx.mtx_model_sizes(d, w.shards, w.shard_batch)
    assert P == orc.param_count(w.net.in_shape, layers)
    assert ld >= P and ld % 64 == 0 and ws > 0


def _err(fn, *args):
    kw = {"stream": 0} if fn in (mtx.mtx_average_grads, mtx.mtx_sgd_update,
                                 mtx.mtx_adam_update, mtx.mtx_adagrad_update,
                                 mtx.mtx_train_step) else {}
    with pytest.raises(mtx.MtxError) as e:
        fn(*args, **kw)
    return e.value.code


def test_invalid_networks_are_rejected():
    L = wl.layer_tuples(wl.LENET)
    good = mtx.make_desc((1, 28, 28), L, wl.F32)
    assert _err(mtx.mtx_model_sizes, good, 0, 4) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_model_sizes, good, 4, 0) == mtx.MTX_EINVAL
    bad_last = mtx.make_desc((1, 28, 28), L[:-1], wl.F32)  # ends in FC with ReLU
    assert _err(mtx.mtx_model_sizes, bad_last, 1, 1) == mtx.MTX_EINVAL
    grp = mtx.make_desc((3, 8, 8), [(1, 4, 3, 1, 1, 2, 0), (0, 2, 1, 1, 0, 1, 0)], wl.F32)
    assert _err(mtx.mtx_model_sizes, grp, 1, 1) == mtx.MTX_EINVAL  # 3 channels, 2 groups
    big = mtx.make_desc((1, 4, 4), [(1, 2, 5, 1, 0, 1, 0), (0, 2, 1, 1, 0, 1, 0)], wl.F32)
    assert _err(mtx.mtx_model_sizes, big, 1, 1) == mtx.MTX_EINVAL  # kernel > input
    pool = mtx.make_desc((1, 8, 8), [(2, 0, 17, 1, 0, 1, 0), (0, 2, 1, 1, 0, 1, 0)], wl.F32)
    assert _err(mtx.mtx_model_sizes, pool, 1, 1) == mtx.MTX_EINVAL  # window > 16
    dt = mtx.make_desc((1, 28, 28), L, 7)
    assert _err(mtx.mtx_model_sizes, dt, 1, 1) == mtx.MTX_EINVAL
    kind = mtx.make_desc((1, 8, 8), [(9, 2, 1, 1, 0, 1, 0), (0, 2, 1, 1, 0, 1, 0)], wl.F32)
    assert _err(mtx.mtx_model_sizes, kind, 1, 1) == mtx.MTX_EINVAL


def test_invalid_residual_and_batch_norm_layers_are_rejected():
    def tup(l):
        if isinstance(l, tuple):
            return l
        return (l.kind, l.out, l.k, l.stride, l.pad, l.groups, int(l.relu))

    base = [wl.conv(8, 3, pad=1), wl.bn(relu=True), wl.conv(8, 3, pad=1), wl.bn(),
            wl.add(1, relu=True), wl.fc(3)]
    good = mtx.make_desc((3, 8, 8), [tup(l) for l in base], wl.F32)
    mtx.mtx_model_sizes(good, 2, 2)

    def code(layers, shape=(3, 8, 8), dt=wl.F32):
        return _err(mtx.mtx_model_sizes, mtx.make_desc(shape, [tup(l) for l in layers], dt), 2, 2)

    L = list(base)
    L[1] = (3, 7, 0, 1, 0, 1, 1)          # BN out differs from its channel count
    assert code(L) == mtx.MTX_EINVAL
    L = list(base)
    L[4] = wl.add(3, relu=True)           # the previous layer is not a shortcut source
    assert code(L) == mtx.MTX_EINVAL
    L = list(base)
    L[4] = wl.add(5)                      # not an earlier layer
    assert code(L) == mtx.MTX_EINVAL
    shape = [wl.conv(8, 3, pad=1), wl.conv(8, 3), wl.add(0), wl.fc(2)]  # 8x8 vs 6x6
    assert code(shape) == mtx.MTX_EINVAL
    twice = base[:5] + [wl.conv(8, 3, pad=1), wl.add(1), wl.fc(3)]   # layer 1 added twice
    assert code(twice) == mtx.MTX_EINVAL
    wide = [wl.fc(300), wl.bn(), wl.fc(2)]  # 300 channels, not a multiple of 8 (bf16)
    assert code(wide, (4, 1, 1), wl.BF16) == mtx.MTX_EUNSUPPORTED


def test_update_argument_errors_need_no_device():
    g = np.zeros(64, np.float32)
    w = np.zeros(16, np.float32)
    a = np.zeros(16, np.float32)
    assert _err(mtx.mtx_average_grads, g, 0, 16, 16, a) == mtx.MTX_EINVAL       # R < 1
    assert _err(mtx.mtx_average_grads, g, 4, 0, 16, a) == mtx.MTX_EINVAL       # n == 0
    assert _err(mtx.mtx_average_grads, g, 4, 16, 8, a) == mtx.MTX_EINVAL       # ld < n
    assert _err(mtx.mtx_average_grads, None, 4, 16, 16, a) == mtx.MTX_EINVAL   # NULL
    assert _err(mtx.mtx_average_grads, g, 4, 16, 16, g[8:]) == mtx.MTX_EINVAL  # overlap
    assert _err(mtx.mtx_sgd_update, w, None, g, 4, 16, 16, 0.1, 0.9, None) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_sgd_update, w, w, g, 4, 16, 16, 0.1, 0.9, None) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_sgd_update, w, None, g, 4, 16, 16, float("nan"), 0.0, None) == mtx.MTX_EINVAL
    mis = g.ctypes.data + 2
    assert _err(mtx.mtx_average_grads, mis, 1, 4, 4, a) == mtx.MTX_EINVAL       # misaligned


def test_adaptive_update_argument_errors_need_no_device():
    g = np.zeros(64, np.float32)
    w, m, v = (np.zeros(16, np.float32) for _ in range(3))
    ok = (0.001, 0.9, 0.999, 1e-8, 1)
    assert _err(mtx.mtx_adam_update, w, None, v, g, 4, 16, 16, *ok) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_adam_update, w, m, m, g, 4, 16, 16, *ok) == mtx.MTX_EINVAL     # m = v
    assert _err(mtx.mtx_adam_update, w, m, v, g, 4, 16, 16, 0.001, 1.0, 0.999, 1e-8, 1) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_adam_update, w, m, v, g, 4, 16, 16, 0.001, 0.9, -0.1, 1e-8, 1) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_adam_update, w, m, v, g, 4, 16, 16, 0.001, 0.9, 0.999, -1.0, 1) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_adam_update, w, m, v, g, 4, 16, 16, 0.001, 0.9, 0.999, 1e-8, 0) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_adam_update, w, m, v, g, 4, 16, 8, *ok) == mtx.MTX_EINVAL      # ld < n
    assert _err(mtx.mtx_adam_update, w, m, g[4:], g, 4, 16, 16, *ok) == mtx.MTX_EINVAL  # overlap
    assert _err(mtx.mtx_adagrad_update, w, None, g, 4, 16, 16, 0.1, 1e-10) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_adagrad_update, w, w, g, 4, 16, 16, 0.1, 1e-10) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_adagrad_update, w, m, g, 0, 16, 16, 0.1, 1e-10) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_adagrad_update, w, m, g, 4, 16, 16, float("inf"), 1e-10) == mtx.MTX_EINVAL


def test_model_call_errors_need_no_device():
    assert _err(mtx.mtx_train_step, None, 16, 16, 0.1, 0.0) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_set_optimizer, None, mtx.MTX_OPT_ADAM) == mtx.MTX_EINVAL
    assert _err(mtx.mtx_get_params, None, np.zeros(4, np.float32)) == mtx.MTX_EINVAL
    L = wl.layer_tuples(wl.MLP)
    d = mtx.make_desc((784, 1, 1), L, wl.F32)
    bufs = mtx.mtx_buffers(0, 0, 0, 0, 0, 0)
    h = C.c_void_p()
    rc = mtx.lib().mtx_init_model(C.byref(d), 2, 32, C.c_uint64(0), C.byref(bufs), None,
                                  C.byref(h))
    assert rc == mtx.MTX_EINVAL and not h.value
    P, ld, ws = mtx.mtx_model_sizes(d, 2, 32)
    small = mtx.mtx_buffers(256, 256 * 4096, 256 * 8192, 256 * 65536, 256 * 1 << 30, ws - 1)
    rc = mtx.lib().mtx_init_model(C.byref(d), 2, 32, C.c_uint64(0), C.byref(small), None,
                                  C.byref(h))
    assert rc == mtx.MTX_ENOMEM
    assert b"workspace too small" in mtx.lib().mtx_last_error()


def test_static_model_takes_no_workspace():
    """mtx_init_model_static refuses a caller workspace before touching a device."""
    L = wl.layer_tuples(wl.LENET)
    d = mtx.make_desc((1, 28, 28), L, wl.F32)
    bufs = mtx.mtx_buffers(16, 16, 16, 16, 256, 1024)
    h = C.c_void_p()
    rc = mtx.lib().mtx_init_model_static(C.byref(d), 1, 1, C.c_uint64(0), C.byref(bufs), None,
                                         C.byref(h))
    assert rc == mtx.MTX_EINVAL and not h.value
    assert b"no workspace" in mtx.lib().mtx_last_error()
