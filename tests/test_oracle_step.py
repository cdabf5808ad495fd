"""Pins of the oracle's training step: torch float64 autograd on whole networks, central finite
differences, closed forms, and the synchronous-SGD invariant.  CPU only."""
import math

import numpy as np
import pytest

from oracle import oracle as orc
from paper_1704_04560_amd import workloads as wl
from tests import torch_ref


def _tiny_net():
    """One of each layer type: grouped strided padded conv + ReLU, overlapping 3/2 pool, 1x1
    conv, FC + ReLU, FC."""
    layers = [wl.conv(4, 3, stride=2, pad=1, groups=2, relu=True), wl.maxpool(3, 2),
              wl.conv(3, 1), wl.fc(5, relu=True), wl.fc(4)]
    net = wl.Net("tiny", (2, 11, 11), tuple(layers), wl.F32, "normal")
    return net, wl.layer_tuples(net)


def _rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


NETS = {
    "mlp": (wl.MLP, 64, 2),
    "lenet": (wl.LENET, 8, 4),
    "cifar": (wl.CIFAR, 2, 2),
    "tiny": (None, 6, 3),
}


@pytest.mark.parametrize("name", list(NETS))
def test_step_matches_torch_autograd(name):
    net, B, R = NETS[name]
    if net is None:
        net, layers = _tiny_net()
    else:
        layers = wl.layer_tuples(net)
    geo = orc.geometry(net.in_shape, layers)
    P = orc.param_count(net.in_shape, layers)
    w = orc.init_glorot(net.in_shape, layers, seed=3)
    # non-zero biases so that they are exercised
    g = np.random.default_rng(11)
    for gg in geo:
        if gg["b_len"]:
            w[gg["b_off"]:gg["b_off"] + gg["b_len"]] = g.normal(0, 0.1, gg["b_len"])
    x, y = wl.make_batch(net, B, seed=5)
    v = wl.make_velocity(P, seed=5)
    res = orc.train_step(net.in_shape, layers, R, x, y, w, v, 0.01, 0.9, prec="exact",
                         want_acts=True)
    gref, lref = torch_ref.shard_grads(layers, geo, w, x, y, R)
    for r in range(R):
        assert abs(res.shard_loss[r] - lref[r]) <= 1e-6 * abs(lref[r])
        assert _rel(res.grads[r], gref[r]) < 2e-7
    assert abs(res.loss - np.mean(lref)) <= 1e-12 * abs(np.mean(lref))
    assert _rel(res.gavg, gref.mean(axis=0)) < 2e-7
    # forward activations of every layer
    import torch
    _, acts = torch_ref.forward(layers, geo, torch.as_tensor(w, dtype=torch.float64),
                                torch.as_tensor(x, dtype=torch.float64))
    off = 0
    for a in acts:
        n = a.numel()
        ours = res.acts[off:off + n]
        assert _rel(ours, a.detach().numpy().ravel()) < 1e-7
        off += n


@pytest.mark.slow
def test_alexnet_step_matches_torch_autograd():
    net = wl.ALEXNET
    layers = wl.layer_tuples(net)
    geo = orc.geometry(net.in_shape, layers)
    assert orc.param_count(net.in_shape, layers) == 60_965_224
    w = orc.init_glorot(net.in_shape, layers, seed=1)
    x, y = wl.make_batch(net, 2, seed=2)
    res = orc.train_step(net.in_shape, layers, 2, x, y, w, None, 0.01, 0.0, prec="exact")
    gref, lref = torch_ref.shard_grads(layers, geo, w, x, y, 2)
    for r in range(2):
        for gg in geo:
            if gg["w_len"]:
                sl = slice(gg["w_off"], gg["b_off"] + gg["b_len"])
                assert _rel(res.grads[r][sl], gref[r][sl]) < 2e-7
        assert abs(res.shard_loss[r] - lref[r]) <= 1e-6 * abs(lref[r])


def test_finite_differences():
    net, layers = _tiny_net()
    P = orc.param_count(net.in_shape, layers)
    w = orc.init_glorot(net.in_shape, layers, seed=7)
    w += np.random.default_rng(1).normal(0, 0.05, P).astype(np.float32)
    x, y = wl.make_batch(net, 4, seed=9)

    def run(wv):
        return orc.train_step(net.in_shape, layers, 2, x, y, wv, None, 0.0, 0.0, prec="exact",
                              want_grads=False, want_decisions=True)

    base = run(w)
    idx = np.random.default_rng(2).choice(P, size=60, replace=False)
    checked = 0
    for i in idx:
        h = 1e-5
        wp, wm = w.copy(), w.copy()
        wp[i] += h
        wm[i] -= h
        rp, rm = run(wp), run(wm)
        # skip coordinates whose perturbation moves a ReLU or pooling decision (a kink)
        if not (np.array_equal(rp.pool_argmax, base.pool_argmax) and
                np.array_equal(rm.pool_argmax, base.pool_argmax) and
                np.array_equal(rp.relu_mask, base.relu_mask) and
                np.array_equal(rm.relu_mask, base.relu_mask)):
            continue
        delta = float(wp[i]) - float(wm[i])
        fd = (rp.loss - rm.loss) / delta
        g = float(base.gavg[i])
        assert abs(fd - g) <= 1e-6 * max(1.0, abs(g)) + 1e-7, (i, fd, g)
        checked += 1
    assert checked >= 40


def test_single_linear_softmax_closed_form():
    """One FC layer followed by softmax cross-entropy: dW = (P - Y)^T X / N, db = 1^T (P - Y) / N."""
    N, IN, NC = 12, 7, 5
    net = wl.Net("lin", (IN, 1, 1), (wl.fc(NC),), wl.F32, "normal")
    layers = wl.layer_tuples(net)
    g = np.random.default_rng(4)
    w = g.normal(0, 0.5, NC * IN + NC).astype(np.float32)
    x, y = wl.make_batch(net, N, seed=4)
    res = orc.train_step(net.in_shape, layers, 1, x, y, w, None, 0.0, 0.0, prec="exact")
    W = w[:NC * IN].reshape(NC, IN).astype(np.float64)
    b = w[NC * IN:].astype(np.float64)
    X = x.reshape(N, IN).astype(np.float64)
    Z = X @ W.T + b
    Pm = np.exp(Z - Z.max(axis=1, keepdims=True))
    Pm /= Pm.sum(axis=1, keepdims=True)
    Y = np.eye(NC)[y]
    dW = (Pm - Y).T @ X / N
    db = (Pm - Y).sum(axis=0) / N
    assert _rel(res.gavg[:NC * IN], dW.ravel()) < 1e-7
    assert _rel(res.gavg[NC * IN:], db) < 1e-7
    loss = np.mean(-np.log(Pm[np.arange(N), y]))
    assert abs(res.loss - loss) < 1e-12


@pytest.mark.parametrize("name", ["mlp", "lenet"])
def test_zero_last_layer_gives_log_c(name):
    net = {"mlp": wl.MLP, "lenet": wl.LENET}[name]
    layers = wl.layer_tuples(net)
    geo = orc.geometry(net.in_shape, layers)
    w = orc.init_glorot(net.in_shape, layers, seed=0)
    last = geo[-1]
    w[last["w_off"]:last["b_off"] + last["b_len"]] = 0.0
    x, y = wl.make_batch(net, 8, seed=0)
    for prec in ("f32", "exact"):
        res = orc.train_step(net.in_shape, layers, 2, x, y, w, None, 0.01, 0.0, prec=prec)
        assert res.loss == math.log(net.num_classes)
        # with the last layer's weights at zero no gradient reaches the earlier layers
        assert np.all(res.gavg[:last["w_off"]] == 0.0)
        # the last bias gradient is mean(softmax - onehot) = 1/C - frequency of each class
        freq = np.bincount(y, minlength=net.num_classes) / len(y)
        assert np.allclose(res.gavg[last["b_off"]:], 1.0 / net.num_classes - freq, atol=1e-7)


@pytest.mark.parametrize("R", [1, 2, 4, 8, 16])
def test_shard_average_equals_full_batch_gradient(R):
    """Synchronous data parallelism (Sec. III-E): the mean of R shard gradients of shard-mean
    losses is the full-batch mean gradient."""
    net = wl.LENET
    layers = wl.layer_tuples(net)
    w = orc.init_glorot(net.in_shape, layers, seed=2)
    x, y = wl.make_batch(net, 16, seed=2)
    full = orc.train_step(net.in_shape, layers, 1, x, y, w, None, 0.01, 0.0, prec="exact")
    part = orc.train_step(net.in_shape, layers, R, x, y, w, None, 0.01, 0.0, prec="exact")
    assert _rel(part.gavg, full.gavg) < 1e-6
    assert abs(part.loss - full.loss) < 1e-12 * abs(full.loss)
    assert _rel(part.w_new, full.w_new) < 1e-7
    if R == 1:
        assert np.array_equal(part.gavg, part.grads[0])


def test_r_shard_trajectory_equals_sequential():
    """Multi-step version of the invariant (the paper's loss curves of default vs 4-GPU
    training coincide): 3 momentum steps with R=4 follow the R=1 trajectory."""
    net = wl.LENET
    layers = wl.layer_tuples(net)
    P = orc.param_count(net.in_shape, layers)
    w1 = orc.init_glorot(net.in_shape, layers, seed=4)
    w4 = w1.copy()
    v1 = np.zeros(P, np.float32)
    v4 = v1.copy()
    for step in range(3):
        x, y = wl.make_batch(net, 8, seed=100 + step)
        a = orc.train_step(net.in_shape, layers, 1, x, y, w1, v1, 0.05, 0.9, prec="exact")
        b = orc.train_step(net.in_shape, layers, 4, x, y, w4, v4, 0.05, 0.9, prec="exact")
        assert abs(a.loss - b.loss) < 1e-6 * abs(a.loss)
        w1, v1, w4, v4 = a.w_new, a.v_new, b.w_new, b.v_new
    assert _rel(w4 - orc.init_glorot(net.in_shape, layers, seed=4),
                w1 - orc.init_glorot(net.in_shape, layers, seed=4)) < 1e-5


def test_bf16_mode_rounds_at_the_stated_points():
    net = wl.CIFAR
    layers = wl.layer_tuples(net)
    w = orc.init_glorot(net.in_shape, layers, seed=1)
    x, y = wl.make_batch(net, 2, seed=1)
    rb = orc.train_step(net.in_shape, layers, 2, x, y, w, None, 0.01, 0.0, prec="bf16",
                        want_acts=True)
    rx = orc.train_step(net.in_shape, layers, 2, x, y, w, None, 0.01, 0.0, prec="exact",
                        want_acts=True)
    geo = orc.geometry(net.in_shape, layers)
    off = 0
    for i, g in enumerate(geo):
        n = int(np.prod(g["out_shape"])) * 2
        a = rb.acts[off:off + n]
        bits = a.view(np.uint32) & 0xFFFF
        if i < len(geo) - 1:
            assert np.all(bits == 0), f"layer {i} output is not bfloat16"
        else:
            assert np.any(bits != 0), "logits are kept in float"
        off += n
    # bfloat16 storage moves max-pool decisions (near-ties within one bf16 step), so early-layer
    # gradients of the two modes differ by up to ~20%; the loss and the last layer barely move.
    last = geo[-1]
    sl = slice(last["w_off"], last["b_off"] + last["b_len"])
    assert _rel(rb.gavg[sl], rx.gavg[sl]) < 2e-2
    assert _rel(rb.gavg, rx.gavg) < 0.5
    assert abs(rb.loss - rx.loss) < 2e-2 * abs(rx.loss)


def _bf16_case(name):
    nets = {"cifar": (wl.CIFAR, 4, 2), "tiny": (_tiny_net()[0], 6, 3),
            "residual": (_residual_net(wl.BF16)[0], 8, 2),
            "projection": (_projection_net(wl.BF16)[0], 8, 2)}
    net, B, R = nets[name]
    layers = wl.layer_tuples(net)
    geo = orc.geometry(net.in_shape, layers)
    w = orc.init_glorot(net.in_shape, layers, seed=3)
    g = np.random.default_rng(11)
    for gg in geo:  # non-zero biases (BN shifts stay 0 at init) so that they are exercised
        if gg["b_len"] and gg["kind"] != 3:
            w[gg["b_off"]:gg["b_off"] + gg["b_len"]] = g.normal(0, 0.1, gg["b_len"])
    x, y = wl.make_batch(net, B, seed=5)
    res = orc.train_step(net.in_shape, layers, R, x, y, w, None, 0.01, 0.0, prec="bf16")
    return net, layers, geo, w, x, y, R, res


def _worst_layer_rel(res, gref, geo, R):
    return max(_rel(res.grads[r][gg["w_off"]:gg["b_off"] + gg["b_len"]],
                    gref[r][gg["w_off"]:gg["b_off"] + gg["b_len"]])
               for r in range(R) for gg in geo if gg["w_len"])


@pytest.mark.parametrize("name", ["cifar", "tiny", "residual", "projection"])
def test_bf16_mode_gradients_match_an_independent_bf16_storage_model(name):
    """Every rounding point of the bf16 mode, the gradient side included, against torch float64
    autograd with bfloat16 storage emulated at exactly those points (torch_ref.forward_bf16):
    x, W, every hidden output, the gradient of the loss with respect to the logits and every
    stored data gradient (a residual source: the next layer's data gradient stored, then the sum
    with the residual path's gradient stored again).  Both evaluate in float64, so they agree to
    the float rounding of the output gradients; a model that omits the loss-gradient rounding or
    the data-gradient roundings disagrees by 1e-3 or more, so a rounding dropped from (or added
    to) the oracle cannot pass."""
    net, layers, geo, w, x, y, R, res = _bf16_case(name)
    gref, lref = torch_ref.shard_grads_bf16(layers, geo, w, x, y, R)
    for r in range(R):
        assert abs(res.shard_loss[r] - lref[r]) <= 1e-6 * abs(lref[r])
    assert _worst_layer_rel(res, gref, geo, R) < 1e-6
    for kw in ({"round_grads": False}, {"round_loss_grad": False}):
        gmiss, _ = torch_ref.shard_grads_bf16(layers, geo, w, x, y, R, **kw)
        assert _worst_layer_rel(res, gmiss, geo, R) > 1e-4, kw


def test_pool_hint_accepts_only_ties_within_the_error_bound():
    # an input with exact ties inside the pooling windows of a conv-free net
    layers = [wl.maxpool(2, 2), wl.fc(3)]
    net = wl.Net("pooltie", (1, 4, 4), tuple(layers), wl.F32, "normal")
    lt = wl.layer_tuples(net)
    x = np.zeros((2, 1, 4, 4), np.float32)
    x[:, 0] = np.array([[1, 1, 0, 2], [0, 0, 1, 0], [3, 0, 0, 0], [0, 3, 5, 5]], np.float32)
    y = np.array([0, 1], np.int32)
    w = np.random.default_rng(0).normal(0, 1, orc.param_count(net.in_shape, lt)).astype(np.float32)
    base = orc.train_step(net.in_shape, lt, 1, x, y, w, None, 0.0, 0.0, want_decisions=True)
    assert list(base.pool_argmax[:4]) == [0, 1, 0, 2]
    # window 0 has a tie between elements 0 and 1: the hint is a valid alternative
    hint = np.full(base.pool_argmax.size, -1, np.int32)
    hint[0] = 1
    alt = orc.train_step(net.in_shape, lt, 1, x, y, w, None, 0.0, 0.0, want_decisions=True,
                         pool_hint=hint)
    assert alt.pool_argmax[0] == 1
    assert np.array_equal(alt.gavg, base.gavg)  # no conv before the pool: same parameter grads
    # window 1 has a unique maximum (2 vs 1): a hint pointing elsewhere must be rejected
    bad = np.full(base.pool_argmax.size, -1, np.int32)
    bad[1] = 0
    with pytest.raises(orc.HintRejected):
        orc.train_step(net.in_shape, lt, 1, x, y, w, None, 0.0, 0.0, pool_hint=bad)


def test_relu_hint_accepts_only_values_within_the_error_bound():
    net = wl.MLP
    layers = wl.layer_tuples(net)
    w = orc.init_glorot(net.in_shape, layers, seed=0)
    x, y = wl.make_batch(net, 4, seed=0)
    base = orc.train_step(net.in_shape, layers, 1, x, y, w, None, 0.0, 0.0, want_decisions=True)
    hint = np.full(base.relu_mask.size, -1, np.int8)
    hint[0] = 1 - base.relu_mask[0]  # flip a decision whose pre-activation is far from zero
    with pytest.raises(orc.HintRejected):
        orc.train_step(net.in_shape, layers, 1, x, y, w, None, 0.0, 0.0, relu_hint=hint)
    same = base.relu_mask.astype(np.int8)
    ok = orc.train_step(net.in_shape, layers, 1, x, y, w, None, 0.0, 0.0, relu_hint=same)
    assert np.array_equal(ok.gavg, base.gavg)


# ---- batch normalisation and residual addition (the building blocks of Table II's ResNet-50) --

def _residual_net(dtype=wl.F32):
    """A residual block with batch normalisation: conv-BN-ReLU-conv-BN, added to the first
    BN-ReLU output, ReLU; then pooling, a 1x1 convolution with BN-ReLU and the classifier."""
    layers = (wl.conv(4, 3, pad=1), wl.bn(relu=True), wl.conv(4, 3, pad=1), wl.bn(),
              wl.add(1, relu=True), wl.maxpool(2, 2), wl.conv(6, 1), wl.bn(relu=True), wl.fc(5))
    net = wl.Net("residual", (3, 8, 8), layers, dtype, "normal")
    return net, wl.layer_tuples(net)


def _projection_net(dtype=wl.F32):
    """A downsampling block with a projection shortcut (strided 1x1 convolution of layer 1's
    output added to the strided main path), then an identity block, pooling and the classifier."""
    layers = (wl.conv(4, 3, pad=1), wl.bn(relu=True),
              wl.conv(8, 3, stride=2, pad=1), wl.bn(), wl.addp(1, 8, stride=2, relu=True),
              wl.conv(8, 3, pad=1), wl.bn(), wl.add(4, relu=True),
              wl.maxpool(2, 2), wl.fc(5))
    net = wl.Net("projection", (3, 8, 8), layers, dtype, "normal")
    return net, wl.layer_tuples(net)


def _perturbed_params(net, layers, seed):
    """Glorot weights (BN: gamma = 1, beta = 0) moved off their initial values, so that every
    parameter, the BN scales and shifts included, takes part."""
    geo = orc.geometry(net.in_shape, layers)
    w = orc.init_glorot(net.in_shape, layers, seed=seed)
    g = np.random.default_rng(seed + 1)
    for gg in geo:
        if gg["kind"] == 3:
            w[gg["w_off"]:gg["w_off"] + gg["w_len"]] = g.uniform(0.5, 1.5, gg["w_len"])
        if gg["b_len"]:
            w[gg["b_off"]:gg["b_off"] + gg["b_len"]] = g.normal(0, 0.1, gg["b_len"])
    return geo, w


@pytest.mark.parametrize("R", [1, 2])
@pytest.mark.parametrize("netf", ["residual", "projection"])
def test_residual_bn_step_matches_torch_autograd(R, netf):
    """Every shard's loss and gradient against torch float64 autograd (F.batch_norm in training
    mode over the shard's samples, tensor addition for the residual, F.conv2d with a 1x1 kernel
    and the stride for the projection shortcut)."""
    net, layers = _residual_net() if netf == "residual" else _projection_net()
    geo, w = _perturbed_params(net, layers, 3)
    x, y = wl.make_batch(net, 6 * R, seed=5)
    res = orc.train_step(net.in_shape, layers, R, x, y, w, None, 0.01, 0.0, prec="exact")
    gref, lref = torch_ref.shard_grads(layers, geo, w, x, y, R)
    for r in range(R):
        assert abs(res.shard_loss[r] - lref[r]) <= 1e-6 * abs(lref[r])
        assert _rel(res.grads[r], gref[r]) < 2e-7
        for gg in geo:  # every parameter tensor on its own, the BN ones included
            sl = slice(gg["w_off"], gg["b_off"] + gg["b_len"])
            if gg["w_len"]:
                assert _rel(res.grads[r][sl], gref[r][sl]) < 1e-6, gg


@pytest.mark.parametrize("netf", ["residual", "projection"])
def test_residual_bn_finite_differences(netf):
    net, layers = _residual_net() if netf == "residual" else _projection_net()
    geo, w = _perturbed_params(net, layers, 7)
    P = w.size
    x, y = wl.make_batch(net, 6, seed=9)

    def run(wv):
        return orc.train_step(net.in_shape, layers, 2, x, y, wv, None, 0.0, 0.0, prec="exact",
                              want_grads=False, want_decisions=True)

    base = run(w)
    checked = 0
    for i in np.random.default_rng(2).choice(P, size=80, replace=False):
        h = 1e-5
        wp, wm = w.copy(), w.copy()
        wp[i] += h
        wm[i] -= h
        rp, rm = run(wp), run(wm)
        if not (np.array_equal(rp.pool_argmax, base.pool_argmax) and
                np.array_equal(rm.pool_argmax, base.pool_argmax) and
                np.array_equal(rp.relu_mask, base.relu_mask) and
                np.array_equal(rm.relu_mask, base.relu_mask)):
            continue
        fd = (rp.loss - rm.loss) / (float(wp[i]) - float(wm[i]))
        g = float(base.gavg[i])
        assert abs(fd - g) <= 1e-6 * max(1.0, abs(g)) + 1e-7, (i, fd, g)
        checked += 1
    assert checked >= 50


def test_bias_before_batch_norm_has_zero_gradient():
    """Batch normalisation removes any per-channel constant from its input, so the bias of the
    convolution that feeds it cannot change the loss: its gradient vanishes (to rounding)."""
    net, layers = _residual_net()
    geo, w = _perturbed_params(net, layers, 11)
    x, y = wl.make_batch(net, 8, seed=12)
    res = orc.train_step(net.in_shape, layers, 2, x, y, w, None, 0.0, 0.0, prec="exact")
    for li in (0, 2, 6):  # the convolutions followed by BN
        gg = geo[li]
        gb = res.grads[:, gg["b_off"]:gg["b_off"] + gg["b_len"]]
        gw = res.grads[:, gg["w_off"]:gg["w_off"] + gg["w_len"]]
        assert np.abs(gb).max() <= 1e-6 * np.abs(gw).max(), li


def test_shard_statistics_make_the_average_differ_from_the_full_batch_gradient():
    """With batch normalisation each replica normalises by its own shard's statistics, so the
    average of the R shard gradients is not the gradient of the full batch (unlike the networks
    without it, test_shard_average_equals_full_batch_gradient); without BN the residual network
    keeps that identity."""
    net, layers = _residual_net()
    geo, w = _perturbed_params(net, layers, 13)
    x, y = wl.make_batch(net, 8, seed=14)
    r4 = orc.train_step(net.in_shape, layers, 4, x, y, w, None, 0.0, 0.0, prec="exact")
    r1 = orc.train_step(net.in_shape, layers, 1, x, y, w, None, 0.0, 0.0, prec="exact")
    assert _rel(r4.gavg, r1.gavg) > 1e-3
    plain = tuple(l for l in layers if l[0] != 3)
    plain = tuple((4, 0, 0, 1, 0, 1, t[6]) if t[0] == 4 else t for t in plain)  # src 1 -> 0
    P = orc.param_count(net.in_shape, plain)
    wp = orc.init_glorot(net.in_shape, plain, seed=15)
    p4 = orc.train_step(net.in_shape, plain, 4, x, y, wp, None, 0.0, 0.0, prec="exact")
    p1 = orc.train_step(net.in_shape, plain, 1, x, y, wp, None, 0.0, 0.0, prec="exact")
    assert P == wp.size and _rel(p4.gavg, p1.gavg) < 1e-6  # float rounding of each shard


def test_projection_shortcut_layers_are_validated():
    net, layers = _projection_net()
    orc.param_count(net.in_shape, layers)
    bad_out = list(layers)
    bad_out[4] = (5, 6, 1, 2, 0, 1, 1)  # out must be this layer's channel count (8)
    bad_stride = list(layers)
    bad_stride[4] = (5, 8, 1, 1, 0, 1, 1)  # stride 1 maps 8x8 to 8x8, not to 4x4
    bad_pad = list(layers)
    bad_pad[4] = (5, 8, 1, 2, 1, 1, 1)
    bad_src = list(layers)
    bad_src[4] = (5, 8, 3, 2, 0, 1, 1)  # the previous layer is not a valid source
    for L in (bad_out, bad_stride, bad_pad, bad_src):
        with pytest.raises(ValueError):
            orc.param_count(net.in_shape, L)
    geo = orc.geometry(net.in_shape, layers)
    assert geo[4]["w_len"] == 8 * 4 and geo[4]["b_len"] == 8
    assert orc.param_count(net.in_shape, layers) == geo[-1]["b_off"] + geo[-1]["b_len"]


def test_residual_bn_layers_are_validated():
    ok = [wl.layer_tuples(_residual_net()[0])]
    orc.param_count((3, 8, 8), ok[0])
    bad_src = list(ok[0])
    bad_src[4] = (4, 0, 3, 1, 0, 1, 1)  # the previous layer is not a valid source
    bad_shape = [wl.layer_tuples(wl.Net("x", (3, 8, 8), (wl.conv(4, 3, pad=1), wl.conv(4, 3),
                                                         wl.add(0), wl.fc(2)), wl.F32, "normal"))]
    bad_bn = list(ok[0])
    bad_bn[1] = (3, 7, 0, 1, 0, 1, 1)  # BN out must equal its channel count
    for L in (bad_src, bad_shape[0], bad_bn):
        with pytest.raises(ValueError):
            orc.param_count((3, 8, 8), L)
