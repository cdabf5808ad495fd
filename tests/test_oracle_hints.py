"""The oracle's check of decision hints rejects wrong decisions at every depth.  CPU only.

The GPU's max-pool and ReLU decisions are handed to the oracle only where they differ from the
oracle's own, and the oracle admits such a hint only inside a window that does not grow with
depth (the parity tolerance times the layer's scale, capped further by the rigorous forward error
bound).  These tests plant wrong decisions on the CPU -- the oracle's own decisions with the
deepest pooling layer or the deepest ReLU replaced -- at the sizes of the GPU parity tests of the
deep networks, and check that the oracle refuses them, in bf16 and in fp32:
  - every window of the deepest pooling layer forced to its first element;
  - every unit of the deepest ReLU forced to pass;
  - one window alone, the one whose forced gap is the median of the changed windows;
  - one unit alone, the blocked unit whose pre-activation is the median of the blocked ones;
and, as a control that the window is not empty, that the blocked unit closest to zero may be
passed in bf16 (exact ties, the fp32 control, are covered by the tests of the step).
"""
import numpy as np
import pytest

from oracle import oracle as orc
from paper_1704_04560_amd import workloads as wl
from tests import parity

# (network, R, shard batch) at the sizes of the GPU parity tests of the deep networks
CASES = {
    "cifar-bf16": (wl.CIFAR, 8, 2),
    "alexnet-bf16": (wl.ALEXNET, 4, 1),
    "resnet-bf16": (wl.RESNET, 2, 2),
    "resnet-f32": (wl.Net("resnet-f32", wl.RESNET.in_shape, wl.RESNET.layers, wl.F32, "normal"), 2, 2),
    "lenet-bf16": (wl.Net("lenet-bf16", wl.LENET.in_shape, wl.LENET.layers, wl.BF16, "uniform"), 4, 8),
}

_cache = {}


def _base(name):
    """The oracle's own step (decisions and stored outputs) on the case's seeded inputs."""
    if name not in _cache:
        net, R, Nb = CASES[name]
        layers = wl.layer_tuples(net)
        prec = "bf16" if net.dtype == wl.BF16 else "f32"
        w = orc.init_glorot(net.in_shape, layers, 7)
        x, y = wl.make_batch(net, R * Nb, seed=7)
        res = orc.train_step(net.in_shape, layers, R, x, y, w, None, 0.0, 0.0, prec=prec,
                             want_grads=False, want_acts=True, want_decisions=True)
        _cache[name] = (net, layers, prec, R, Nb, w, x, y, res)
    return _cache[name]


def _segment(net, layers, B, kind, which=-1):
    segs = [s for s in parity.decision_layers(net.in_shape, layers, B) if s[1] == kind]
    return segs[which]


def _run(name, pool_hint=None, relu_hint=None):
    net, layers, prec, R, Nb, w, x, y, _ = _base(name)
    return orc.train_step(net.in_shape, layers, R, x, y, w, None, 0.0, 0.0, prec=prec,
                          want_grads=False, pool_hint=pool_hint, relu_hint=relu_hint)


def _pool_gaps(name):
    """Per window of the deepest pooling layer (shard 0): maximum minus the first element, from
    the oracle's stored pool input."""
    net, layers, prec, R, Nb, w, x, y, res = _base(name)
    geo = orc.geometry(net.in_shape, layers)
    li, _, off, n, _ = _segment(net, layers, R * Nb, "pool")
    c, h, wd = geo[li]["in_shape"]
    s = layers[li][3]
    aoff = sum(int(np.prod(g["out_shape"])) * R * Nb for g in geo[:li - 1])
    a = res.acts[aoff:aoff + Nb * c * h * wd].reshape(Nb, c, h, wd).astype(np.float64)
    oc, oh, ow = geo[li]["out_shape"]
    first = a[:, :, 0:(oh - 1) * s + 1:s, 0:(ow - 1) * s + 1:s][:, :, :oh, :ow]
    pooled = res.acts[sum(int(np.prod(g["out_shape"])) * R * Nb for g in geo[:li]):][:Nb * oc * oh * ow]
    return (pooled.reshape(Nb, oc, oh, ow) - first).ravel(), off, n


@pytest.mark.parametrize("name", list(CASES))
def test_deepest_pool_forced_to_first_element_is_rejected(name):
    net, layers, prec, R, Nb, w, x, y, res = _base(name)
    _, _, off, n, _ = _segment(net, layers, R * Nb, "pool")
    ph = np.full(res.pool_argmax.size, -1, np.int32)
    ph[off:off + n] = 0
    changed = int((res.pool_argmax[off:off + n] != 0).sum())
    assert changed > n // 10  # a real plant: many decisions move
    with pytest.raises(orc.HintRejected):
        _run(name, pool_hint=ph)


@pytest.mark.parametrize("name", list(CASES))
def test_deepest_relu_forced_on_is_rejected(name):
    net, layers, prec, R, Nb, w, x, y, res = _base(name)
    _, _, off, n, _ = _segment(net, layers, R * Nb, "relu")
    rh = np.full(res.relu_mask.size, -1, np.int8)
    rh[off:off + n] = 1
    assert int((res.relu_mask[off:off + n] == 0).sum()) > n // 10
    with pytest.raises(orc.HintRejected):
        _run(name, relu_hint=rh)


@pytest.mark.parametrize("name", list(CASES))
def test_one_median_pool_window_forced_is_rejected(name):
    """One wrong window alone (not a count limit): the first element of the window whose gap to
    the maximum is the median gap among the windows it would change."""
    net, layers, prec, R, Nb, w, x, y, res = _base(name)
    gaps, off, n = _pool_gaps(name)
    am = res.pool_argmax[off:off + gaps.size]
    cand = np.flatnonzero((am != 0) & (gaps > 0))
    t = cand[np.argsort(gaps[cand])[cand.size // 2]]
    ph = np.full(res.pool_argmax.size, -1, np.int32)
    ph[off + t] = 0
    with pytest.raises(orc.HintRejected):
        _run(name, pool_hint=ph)


def _preactivations(name):
    """Pre-activations of the deepest ReLU layer for shard 0's samples: the same network with
    that layer's ReLU removed stores them as its output (the layers below are unchanged)."""
    net, layers, prec, R, Nb, w, x, y, res = _base(name)
    li, _, off, n, _ = _segment(net, layers, R * Nb, "relu")
    lt = list(layers)
    lt[li] = tuple(lt[li][:6]) + (0,)
    geo = orc.geometry(net.in_shape, lt)
    r1 = orc.train_step(net.in_shape, lt, 1, x[:Nb], y[:Nb], w, None, 0.0, 0.0, prec=prec,
                        want_grads=False, want_acts=True)
    aoff = sum(int(np.prod(g["out_shape"])) * Nb for g in geo[:li])
    z = r1.acts[aoff:aoff + int(np.prod(geo[li]["out_shape"])) * Nb].astype(np.float64)
    return z, off


@pytest.mark.parametrize("name", list(CASES))
def test_one_median_relu_unit_forced_on_is_rejected_and_one_near_zero_is_admitted(name):
    net, layers, prec, R, Nb, w, x, y, res = _base(name)
    z, off = _preactivations(name)
    blocked = np.flatnonzero(z < 0)
    order = blocked[np.argsort(-z[blocked])]  # closest to zero first
    rh = np.full(res.relu_mask.size, -1, np.int8)
    med = order[order.size // 2]
    rh[off + med] = 1
    with pytest.raises(orc.HintRejected):
        _run(name, relu_hint=rh)
    if prec == "bf16":  # the nearest to zero of thousands of units: far inside the window
        rh[off + med] = -1
        rh[off + order[0]] = 1
        _run(name, relu_hint=rh)
