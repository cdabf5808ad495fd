"""GPU parity of mtx_train_step against the CPU oracle, through the C ABI.

Every step starts both sides from the same state (the oracle's weights and velocity are copied
into the model before the step), runs one step on the same seeded batch, and compares the loss,
every shard's per-layer weight and bias gradients, the averaged gradient, the velocity, the
weight update and every layer's stored output.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_1704_04560_amd import mtx
from paper_1704_04560_amd import workloads as wl
from tests import parity

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def run_case(tag, net, R, Nb, steps, seed, lr, mu, check_acts=True, tol=None, configure=None):
    layers = wl.layer_tuples(net)
    geo = orc.geometry(net.in_shape, layers)
    prec = "bf16" if net.dtype == wl.BF16 else "f32"
    tol = parity.TOL[net.dtype] if tol is None else tol
    _say(f"[case] {tag}: B={R * Nb} R={R} dtype={prec} steps={steps}")
    model = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=seed)
    if configure is not None:
        configure(model)
    w = orc.init_glorot(net.in_shape, layers, seed)
    v = np.zeros_like(w)
    wg, vg = model.get_params()
    assert np.array_equal(wg.view(np.uint32), w.view(np.uint32)), "initial weights differ"
    assert np.all(vg == 0)
    loss_dev = torch.zeros(1, device="cuda")
    hinted = 0
    for step in range(steps):
        x, y = wl.make_batch(net, R * Nb, seed=seed * 1000 + step)
        model.set_params(w, v)
        model.train_step(torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), lr, mu, loss_dev)
        torch.cuda.synchronize()
        gp, gr = parity.gpu_decisions(model, geo)
        res, nh = parity.oracle_step_matching(net, layers, R, x, y, w, v if mu else None, lr, mu,
                                              prec, gp, gr, tag=f"{tag} step {step}")
        hinted += nh
        parity.compare_step(model, net, layers, geo, R, res, w, v, mu, tol, float(loss_dev.item()),
                            check_acts=check_acts)
        w = res.w_new
        if mu:
            v = res.v_new
    _say(f"[case] {tag}: ok ({hinted} hinted decisions)")
    model.close()


def _tiny(dtype):
    layers = (wl.conv(6, 3, pad=1, relu=True), wl.conv(8, 3, stride=2, pad=1, groups=2, relu=True),
              wl.maxpool(3, 2), wl.conv(5, 1), wl.fc(7, relu=True), wl.fc(4))
    return wl.Net("tiny", (3, 13, 11), layers, dtype, "normal")


def test_mlp_config():
    run_case("mlp", wl.MLP, 2, 32, 3, 1, 0.01, 0.0)


def test_mlp_with_momentum():
    run_case("mlp-momentum", wl.MLP, 2, 32, 3, 2, 0.01, 0.9)


def test_lenet_small():
    run_case("lenet-small", wl.LENET, 4, 4, 3, 3, 0.01, 0.9)


def test_lenet_config():
    run_case("lenet", wl.LENET, 4, 64, 2, 4, 0.01, 0.9)


def _residual(dtype):
    """A residual block with batch normalisation (conv-BN-ReLU-conv-BN + shortcut, ReLU), then
    pooling, a 1x1 convolution with BN-ReLU and the classifier."""
    layers = (wl.conv(8, 3, pad=1), wl.bn(relu=True), wl.conv(8, 3, pad=1), wl.bn(),
              wl.add(1, relu=True), wl.maxpool(2, 2), wl.conv(16, 1), wl.bn(relu=True), wl.fc(5))
    return wl.Net("residual", (3, 8, 8), layers, dtype, "normal")


def _residual_edges(dtype):
    """Batch normalisation of the input itself, a shortcut whose source is a pooling output,
    and batch normalisation after a fully connected layer (one position per channel)."""
    layers = (wl.bn(), wl.conv(8, 3, pad=1, relu=True), wl.maxpool(2, 2),
              wl.conv(8, 3, pad=1), wl.bn(relu=True), wl.add(2), wl.fc(12), wl.bn(relu=True),
              wl.fc(3))
    return wl.Net("residual-edges", (3, 8, 8), layers, dtype, "normal")


def _tiny_unpadded(dtype):
    """Unpadded convolutions below the first layer, grouped and strided: their data gradient
    goes through the col + col2im path."""
    layers = (wl.conv(4, 3, pad=1, relu=True), wl.conv(6, 5, stride=2, groups=2, relu=True),
              wl.conv(4, 3, groups=2), wl.fc(5, relu=True), wl.fc(3))
    return wl.Net("tiny2", (2, 11, 11), layers, dtype, "normal")


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_every_layer_type(dtype):
    run_case(f"tiny-{dtype}", _tiny(dtype), 3, 5, 2, 5, 0.05, 0.9)


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_unpadded_grouped_strided_convolutions(dtype):
    run_case(f"tiny2-{dtype}", _tiny_unpadded(dtype), 2, 3, 2, 6, 0.05, 0.9)


def _tiny_pools(dtype):
    """Pooling windows other than 2/2 and 3/2 (overlapping and not, with and without a ReLU
    below), and a 3/2 window feeding a fully connected layer."""
    layers = (wl.conv(4, 3, pad=1, relu=True), wl.maxpool(2, 1), wl.conv(6, 3), wl.maxpool(3, 3),
              wl.conv(8, 1, relu=True), wl.maxpool(3, 2), wl.fc(3))
    return wl.Net("tiny3", (3, 17, 15), layers, dtype, "normal")


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_pool_windows_and_strides(dtype):
    run_case(f"tiny3-{dtype}", _tiny_pools(dtype), 2, 3, 2, 10, 0.05, 0.9)


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_pool_before_fc_with_an_odd_channel_group(dtype):
    """A 3/2 pooling of 24 channels to 3 x 3 positions feeding a fully connected layer: the
    pooled output is NCHW, a block takes all 24 channels (not a power of two), and its 216
    outputs start at offsets that are not 16-byte aligned in the argmax tensor."""
    layers = (wl.conv(24, 3, pad=1, relu=True), wl.maxpool(3, 2), wl.fc(5))
    net = wl.Net("pool-odd", (3, 7, 7), layers, dtype, "normal")
    run_case(f"pool-odd-{dtype}", net, 2, 3, 2, 12, 0.05, 0.9)


def _single_channel(dtype, oc, k, pad, relu):
    """One input channel into a small-window first convolution: the shape the direct
    first-convolution kernels take (ragged image, several output-channel counts and windows)."""
    layers = (wl.conv(oc, k, pad=pad, relu=relu), wl.maxpool(2, 2), wl.conv(6, 3, relu=True),
              wl.fc(5))
    return wl.Net(f"one-channel-{oc}-{k}", (1, 13, 11), layers, dtype, "normal")


def _sites(model, x, y):
    """Launch-site names of one timed step."""
    loss = torch.zeros(1, device="cuda")
    mtx.mtx_set_timing(model.handle, True)
    mtx.mtx_get_timing(model.handle, reset=True)
    model.train_step(x, y, 0.0, 0.0, loss)
    torch.cuda.synchronize()
    names = {(n, l) for (n, l, k, _) in mtx.mtx_get_timing(model.handle) if k}
    mtx.mtx_set_timing(model.handle, False)
    return names


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("oc,k,pad,relu", [(20, 5, 0, False), (4, 3, 1, True), (32, 3, 0, True),
                                           (16, 7, 3, False), (8, 5, 2, True)])
def test_single_channel_first_convolution(dtype, oc, k, pad, relu):
    net = _single_channel(dtype, oc, k, pad, relu)
    run_case(f"{net.name}-{dtype}", net, 3, 5, 2, 11, 0.05, 0.9)


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("pool_k,pool_s,relu", [(3, 3, True), (2, 1, True), (3, 3, False)])
def test_single_channel_first_convolution_pool_windows(dtype, pool_k, pool_s, relu):
    """The pooling above a direct first convolution: a 3x3/3 window (folded into the direct
    kernels, with ragged rows and columns left over, with and without the ReLU gate) and an
    overlapping 2x2/1 window (not folded: the pooling kernels run)."""
    layers = (wl.conv(8, 5, pad=2, relu=relu), wl.maxpool(pool_k, pool_s), wl.conv(6, 3, relu=True),
              wl.fc(5))
    net = wl.Net(f"one-channel-pool{pool_k}{pool_s}", (1, 14, 13), layers, dtype, "normal")
    run_case(f"{net.name}-{dtype}-{relu}", net, 2, 5, 2, 14, 0.05, 0.9)


def test_first_convolution_takes_the_direct_kernels():
    """LeNet's first layer (one channel, 5x5, 20 outputs) runs on the direct kernels, and a first
    convolution outside their limits (64 outputs of a 7x7 window) on the matrix kernels; with the
    direct kernels, the pooling above needs no backward launch of its own."""
    for net, direct in ((wl.LENET, True), (_single_channel(wl.F32, 64, 7, 3, True), False)):
        layers = wl.layer_tuples(net)
        model = mtx.Model(net.in_shape, layers, net.dtype, 2, 3, seed=1)
        x, y = wl.make_batch(net, 6, seed=1)
        names = _sites(model, torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda())
        model.close()
        assert (("fwd_direct", 0) in names) == direct, names
        assert (("wgrad_direct", 0) in names) == direct, names
        assert (("fwd", 0) in names) != direct, names
        # the 2x2 pooling above hands its gradient to the direct kernel: no pooling backward
        assert (("pool_bwd", 1) in names) != direct, names


def _small_image_dgrad(dtype, k):
    """A convolution below the first layer whose output is a few positions of a small image
    (its data gradient goes through the col tile; in fp32 the tile stays in LDS): ragged row
    tiles and channel ranges, output channel counts that are not multiples of 4, a ReLU mask."""
    if k == 5:
        layers = (wl.conv(23, 3, pad=1, relu=True), wl.conv(13, 5, relu=True), wl.maxpool(2, 2),
                  wl.fc(5))
        return wl.Net("small-dgrad-5", (2, 10, 9), layers, dtype, "normal")
    layers = (wl.conv(30, 3, relu=True), wl.conv(7, 3), wl.fc(4))
    return wl.Net("small-dgrad-3", (1, 9, 9), layers, dtype, "normal")


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
@pytest.mark.parametrize("k", [3, 5])
def test_small_image_data_gradient(dtype, k):
    run_case(f"small-dgrad-{k}-{dtype}", _small_image_dgrad(dtype, k), 3, 4, 2, 13, 0.05, 0.9)


def test_lenet_bf16_reduced_batch():
    net = wl.Net("lenet-bf16", wl.LENET.in_shape, wl.LENET.layers, wl.BF16, "uniform")
    run_case("lenet-bf16", net, 4, 8, 2, 12, 0.01, 0.9)


def test_cifar_shapes_reduced_batch():
    run_case("cifar-B16", wl.CIFAR, 8, 2, 2, 6, 0.01, 0.9)


def test_alexnet_shapes_reduced_batch():
    run_case("alexnet-B4", wl.ALEXNET, 4, 1, 1, 7, 0.01, 0.9, check_acts=False)


@pytest.mark.parametrize("R,Nb", [(1, 1), (1, 7), (3, 5), (16, 1)])
def test_edge_shard_shapes(R, Nb):
    run_case(f"lenet-R{R}-Nb{Nb}", wl.LENET, R, Nb, 1, 8, 0.01, 0.9)


def test_steps_are_deterministic():
    net = wl.LENET
    layers = wl.layer_tuples(net)
    _say("[case] determinism")
    outs = []
    for _ in range(2):
        m = mtx.Model(net.in_shape, layers, net.dtype, 4, 16, seed=9)
        x, y = wl.make_batch(net, 64, seed=9)
        xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
        for _ in range(2):
            m.train_step(xd, yd, 0.01, 0.9)
        w, v = m.get_params()
        outs.append((w, v, m.grads_host()))
        m.close()
    for a, b in zip(outs[0], outs[1]):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_average_is_mean_of_shard_gradients_at_full_alexnet_size():
    """Properties that hold at any size, checked at the full AlexNet size in numpy (no oracle
    call on GPU values): the stored average is the mean of the R stored shard gradients, and
    the update is v' = mu v + avg, w' = w - lr v'."""
    net = wl.ALEXNET
    layers = wl.layer_tuples(net)
    R, Nb = 8, 32
    _say("[case] alexnet full-size step properties")
    m = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=1)
    w0, v0 = m.get_params()
    v0 = wl.make_velocity(m.P, seed=1)
    m.set_params(w0, v0)
    x, y = wl.make_batch(net, R * Nb, seed=1)
    loss = torch.zeros(1, device="cuda")
    m.train_step(torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), 0.01, 0.9, loss)
    torch.cuda.synchronize()
    g = m.grads_host().astype(np.float64)
    avg = m.grad_avg.cpu().numpy()
    parity.assert_tensor_close(avg, g.mean(axis=0), 1e-6, "average")
    w1, v1 = m.get_params()
    v_ref = 0.9 * v0.astype(np.float64) + avg.astype(np.float64)
    parity.assert_tensor_close(v1, v_ref, 1e-6, "velocity")
    parity.assert_update_close(w1, w0.astype(np.float64) - 0.01 * v1.astype(np.float64), w0, 1e-4)
    assert np.isfinite(loss.item()) and abs(loss.item() - np.log(1000)) < 0.5
    m.close()


def _sample_decisions(model, geo, idx):
    """The GPU's pooling and ReLU decisions of the samples idx (oracle layout, concatenated over
    layers), for an oracle run on those samples alone."""
    B = model.B
    pools, relus = [], []
    for i, g in enumerate(geo):
        per = int(np.prod(g["out_shape"]))
        if g["kind"] == 2:
            pools.append(model.pool_argmax(i).astype(np.int32).reshape(B, per)[idx].ravel())
        if g["relu"]:
            relus.append((model.layer_output(i) > 0).astype(np.int8).reshape(B, per)[idx].ravel())
    return (np.concatenate(pools) if pools else np.zeros(0, np.int32),
            np.concatenate(relus) if relus else np.zeros(0, np.int8))


@pytest.mark.parametrize("name", ["cifar", "alexnet"])
def test_full_size_logits_match_oracle_on_sampled_samples(name):
    """The bf16 workloads at their full size, in the launch configuration the benchmark times
    (CIFAR B = 512, AlexNet B = 256, R = 8): a sample's forward pass does not depend on the rest
    of the batch, so the oracle computes the logits of four sampled samples on their own and
    they must match the GPU's stored logits of those samples (decisions near ties taken as the
    GPU took them, within the oracle's error bound)."""
    w = wl.WORKLOADS[name]
    net = w.net
    layers = wl.layer_tuples(net)
    geo = orc.geometry(net.in_shape, layers)
    _say(f"[case] full-size sampled logits {name}")
    model = mtx.Model(net.in_shape, layers, net.dtype, w.shards, w.shard_batch, seed=5)
    wt, _ = model.get_params()
    x, y = wl.make_batch(net, w.batch, seed=5)
    model.train_step(torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), 0.0, 0.0)
    torch.cuda.synchronize()
    idx = np.array([0, w.shard_batch + 7, w.batch // 2 + 3, w.batch - 1])
    gp, gr = _sample_decisions(model, geo, idx)
    res, _ = parity.oracle_step_matching(net, layers, 1, x[idx], y[idx], wt, None, 0.0, 0.0,
                                         "bf16", gp, gr)
    nc = net.num_classes
    logits = model.layer_output(len(geo) - 1).reshape(w.batch, nc)[idx]
    ref = res.acts[-len(idx) * nc:].reshape(len(idx), nc)
    parity.assert_tensor_close(logits, ref, parity.TOL[net.dtype], f"{name} sampled logits")
    model.close()


def _shard_slice(model, geo, r):
    """The GPU's pooling and ReLU decisions and stored outputs of shard r (oracle layout)."""
    Nb = model.Nb
    idx = np.arange(r * Nb, (r + 1) * Nb)
    gp, gr = _sample_decisions(model, geo, idx)
    acts = [model.layer_output(i).reshape(model.B, -1)[idx].ravel() for i in range(len(geo))]
    return gp, gr, acts


@pytest.mark.parametrize("name,shard", [("cifar", 0), ("cifar", 7), ("alexnet", 0),
                                        ("alexnet", 7), ("resnet", 0), ("resnet", 7),
                                        ("bottleneck", 0)])
def test_full_size_shard_gradients_match_oracle(name, shard):
    """The bf16 workloads at their full size in the launch configuration the benchmark times
    (CIFAR B = 512, AlexNet B = 256, the residual network B = 512; R = 8): the whole batch runs on
    the GPU, and the oracle runs shard 0, or shard R - 1, on its own (R = 1, the shard's samples;
    the shard's gradient depends on nothing else, batch normalisation included, whose statistics
    are the shard's).  Every layer's W and b gradient row of that shard, and every stored output
    of its samples, must match at the bf16 bound, parity.RESNET_TOL for the residual network
    (Sec. III-E: each replica's gradient is the sequential gradient of its shard).  The test prints the matrix launches it reached: the
    weight gradients with split reductions and the interleaved schedule, and the data gradients
    at the tile shapes the benchmark runs."""
    w = wl.WORKLOADS[name]
    net = w.net
    layers = wl.layer_tuples(net)
    geo = orc.geometry(net.in_shape, layers)
    tol = parity.RESNET_TOL if name in ("resnet", "bottleneck") else parity.TOL[net.dtype]
    _say(f"[case] full-size shard gradients {name} shard {shard}: B={w.batch} R={w.shards}")
    model = mtx.Model(net.in_shape, layers, net.dtype, w.shards, w.shard_batch, seed=5)
    wt, _ = model.get_params()
    assert np.array_equal(wt.view(np.uint32),
                          orc.init_glorot(net.in_shape, layers, 5).view(np.uint32))
    x, y = wl.make_batch(net, w.batch, seed=5)
    model.train_step(torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), w.lr, w.momentum)
    torch.cuda.synchronize()
    launches = mtx.mtx_get_launches(model.handle)
    grads = model.grads_host()[shard].copy()
    gp, gr, acts = _shard_slice(model, geo, shard)
    model.close()
    torch.cuda.empty_cache()
    seen = sorted({(l["site"], l["tile_rows"], l["tile_cols"], l["splits"], l["flags"])
                   for l in launches})
    _say(f"[launches] {name}: " + ", ".join(f"{s}:{r}x{c}/s{sp}/f{f}" for s, r, c, sp, f in seen))
    Nb = w.shard_batch
    sl = slice(shard * Nb, (shard + 1) * Nb)
    res, _ = parity.oracle_step_matching(net, layers, 1, x[sl], y[sl], wt, None, 0.0, 0.0, "bf16",
                                         gp, gr, tag=f"{name} shard {shard}")
    for gi, g in enumerate(geo):
        if not g["w_len"]:
            continue
        for nm, off, ln in (("W", g["w_off"], g["w_len"]), ("b", g["b_off"], g["b_len"])):
            s_ = slice(off, off + ln)
            if nm == "b" and parity.zero_by_batch_norm(geo, gi):
                wsl = slice(g["w_off"], g["w_off"] + g["w_len"])
                parity._assert_noise(grads[s_], res.grads[0, s_],
                                     float(np.max(np.abs(res.grads[0, wsl]))), tol,
                                     f"layer {gi} b shard {shard}")
                continue
            parity.assert_tensor_close(grads[s_], res.grads[0, s_], tol,
                                       f"{name} layer {gi} {nm} shard {shard}")
    off = 0
    for gi, g in enumerate(geo):
        n = int(np.prod(g["out_shape"])) * Nb
        parity.assert_tensor_close(acts[gi], res.acts[off:off + n], tol,
                                   f"{name} layer {gi} output shard {shard}")
        off += n
    # the launches the benchmark times: split weight gradients with the interleaved schedule
    assert any(l["site"] == "wgrad" and l["splits"] > 1 and l["flags"] & mtx.MTX_GEMM_INTERLEAVED
               for l in launches), seen
    assert any(l["site"] == "dgrad" and l["tile_rows"] * l["tile_cols"] >= 64 * 128
               for l in launches), seen
    if name == "alexnet":
        # conv1's 96 output channels: the 96-row weight-gradient tile with row-along loads
        assert any(l["site"] == "wgrad" and l["tile_rows"] == 96 and l["splits"] > 1
                   for l in launches), seen


@pytest.mark.parametrize("name", ["cifar", "alexnet"])
def test_full_size_shard_count_invariance(name):
    """At the full batch, the weight change of one step does not depend on how the batch is
    split (R = 8 as benchmarked against R = 1 and 2): every launch configuration of the step at
    full size agrees with the others (bf16 bound)."""
    w = wl.WORKLOADS[name]
    net = w.net
    layers = wl.layer_tuples(net)
    _say(f"[case] full-size shard-count invariance {name}")
    x, y = wl.make_batch(net, w.batch, seed=6)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    deltas = {}
    for R in (1, 2, w.shards):
        m = mtx.Model(net.in_shape, layers, net.dtype, R, w.batch // R, seed=6)
        w0, _ = m.get_params()
        m.train_step(xd, yd, w.lr, w.momentum)
        torch.cuda.synchronize()
        w1, _ = m.get_params()
        deltas[R] = w1.astype(np.float64) - w0.astype(np.float64)
        m.close()
        torch.cuda.empty_cache()
    tol = parity.TOL[net.dtype]
    for R in (2, w.shards):
        d, ref = deltas[R], deltas[1]
        assert np.linalg.norm(d - ref) <= tol * np.linalg.norm(ref), R
        assert np.max(np.abs(d - ref)) <= tol * np.max(np.abs(ref)), R


@pytest.mark.parametrize("name", ["lenet", "cifar"])
def test_graph_replay_matches_direct_launches(name):
    """Replaying the captured step gives bit-identical results to enqueuing it directly, on
    every step, with host copies and synchronisations between the replays."""
    net = {"lenet": wl.LENET, "cifar": wl.CIFAR}[name]
    layers = wl.layer_tuples(net)
    R, Nb = (4, 16) if name == "lenet" else (8, 2)
    _say(f"[case] graph replay vs direct {name}")
    a = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=3)
    b = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=3)
    mtx.mtx_set_graph_replay(a.handle, True)
    mtx.mtx_set_graph_replay(b.handle, False)
    x, y = wl.make_batch(net, R * Nb, seed=3)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    la, lb = torch.zeros(1, device="cuda"), torch.zeros(1, device="cuda")
    for step in range(4):
        a.train_step(xd, yd, 0.01, 0.9, la)
        b.train_step(xd, yd, 0.01, 0.9, lb)
        torch.cuda.synchronize()
        wa, va = a.get_params()
        wb, vb = b.get_params()
        assert np.array_equal(wa.view(np.uint32), wb.view(np.uint32)), step
        assert np.array_equal(va.view(np.uint32), vb.view(np.uint32)), step
        assert np.array_equal(a.grads_host().view(np.uint32), b.grads_host().view(np.uint32))
        assert la.item() == lb.item()
    # a new learning rate forces a new capture; results still match
    a.train_step(xd, yd, 0.02, 0.9, la)
    b.train_step(xd, yd, 0.02, 0.9, lb)
    torch.cuda.synchronize()
    assert np.array_equal(a.get_params()[0].view(np.uint32), b.get_params()[0].view(np.uint32))
    a.close()
    b.close()


@pytest.mark.parametrize("name,layerwise", [("lenet", False), ("lenet", True), ("tiny", False),
                                            ("tiny", True),
                                            ("cifar", True), ("alexnet", False),
                                            ("alexnet", True), ("residual", True),
                                            ("resnet", False)])
def test_overlapped_weight_gradients_match_one_stream(name, layerwise):
    """Weight gradients on the second stream (and, with layerwise, each layer's average + update
    on a third stream as soon as its gradients are written) give bit-identical results to the
    one-stream order with one average + update at the end, over several graph-replayed and
    direct steps."""
    net = {"lenet": wl.LENET, "tiny": _tiny(wl.BF16), "cifar": wl.CIFAR,
           "alexnet": wl.ALEXNET, "residual": _residual(wl.BF16), "resnet": wl.RESNET}[name]
    layers = wl.layer_tuples(net)
    R, Nb = {"lenet": (4, 16), "tiny": (3, 5), "cifar": (2, 2), "alexnet": (2, 2),
             "residual": (3, 4), "resnet": (2, 2)}[name]
    _say(f"[case] overlap vs one stream {name} layerwise={layerwise}")
    a = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=4)
    b = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=4)
    mtx.mtx_set_overlap(a.handle, True)
    mtx.mtx_set_layerwise_update(a.handle, layerwise)
    mtx.mtx_set_graph_replay(a.handle, True)
    mtx.mtx_set_overlap(b.handle, False)
    x, y = wl.make_batch(net, R * Nb, seed=4)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    for step in range(3):
        if step == 2:
            mtx.mtx_set_graph_replay(a.handle, False)
        a.train_step(xd, yd, 0.01, 0.9)
        b.train_step(xd, yd, 0.01, 0.9)
        torch.cuda.synchronize()
        assert np.array_equal(a.grads_host().view(np.uint32), b.grads_host().view(np.uint32)), step
        wa, va = a.get_params()
        wb, vb = b.get_params()
        assert np.array_equal(wa.view(np.uint32), wb.view(np.uint32)), step
        assert np.array_equal(va.view(np.uint32), vb.view(np.uint32)), step
        ga, gb = a.grad_avg.cpu().numpy(), b.grad_avg.cpu().numpy()
        assert np.array_equal(ga.view(np.uint32), gb.view(np.uint32)), step
    a.close()
    b.close()


def _wide_fc(dtype):
    """A large fully connected layer (8.4 M parameters, 528 tiles of 128 x 128) that carries
    its own average + update, then a 1.05 M-parameter one (too few 128 x 128 tiles: not fused)
    and a small classifier, whose parameters the stand-alone average + update covers."""
    return wl.Net("wide-fc", (4096, 1, 1), (wl.fc(2048, relu=True), wl.fc(512, relu=True),
                                           wl.fc(10)), dtype, "normal")


@pytest.mark.parametrize("name,R,Nb,mu", [("wide-f32", 2, 8, 0.9), ("wide-bf16", 4, 4, 0.0),
                                           ("alexnet", 2, 2, 0.9), ("alexnet", 8, 1, 0.0),
                                           ("alexnet", 8, 32, 0.9), ("lenet", 4, 16, 0.9)])
def test_fused_fc_update_is_bit_identical(name, R, Nb, mu):
    """Large fully connected layers average and update their own parameters in their
    weight-gradient launch (all R shards of a tile in one block); the shard rows, the average,
    the velocity and the weights are bit-identical to the stand-alone average + update over all
    parameters, with momentum and with plain SGD, over direct and graph-replayed steps.  The
    launch record shows which launches were fused: layers of at least 2^20 parameters with at
    least 512 tiles of 128 x 128 only; at the full AlexNet size too, where the weight gradients
    run on the second stream."""
    net = {"wide-f32": _wide_fc(wl.F32), "wide-bf16": _wide_fc(wl.BF16), "alexnet": wl.ALEXNET,
           "lenet": wl.LENET}[name]
    expect = {"wide-f32": [0], "wide-bf16": [0], "alexnet": [8, 9], "lenet": []}[name]
    layers = wl.layer_tuples(net)
    _say(f"[case] fused fc update {name} R={R} Nb={Nb} mu={mu}")
    a = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=6)
    b = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=6)
    mtx.mtx_set_fused_update(b.handle, False)
    mtx.mtx_set_graph_replay(a.handle, True)
    x, y = wl.make_batch(net, R * Nb, seed=6)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    v0 = a.get_params()[1].copy()
    for step in range(3):
        if step == 2:
            mtx.mtx_set_graph_replay(a.handle, False)
        a.train_step(xd, yd, 0.01, mu)
        b.train_step(xd, yd, 0.01, mu)
        torch.cuda.synchronize()
        assert np.array_equal(a.grads_host().view(np.uint32), b.grads_host().view(np.uint32)), step
        wa, va = a.get_params()
        wb, vb = b.get_params()
        assert np.array_equal(wa.view(np.uint32), wb.view(np.uint32)), step
        assert np.array_equal(va.view(np.uint32), vb.view(np.uint32)), step
        ga, gb = a.grad_avg.cpu().numpy(), b.grad_avg.cpu().numpy()
        assert np.array_equal(ga.view(np.uint32), gb.view(np.uint32)), step
    if mu == 0.0:  # plain SGD leaves v alone
        assert np.array_equal(a.get_params()[1].view(np.uint32), v0.view(np.uint32))
    fused = [l for l in mtx.mtx_get_launches(a.handle) if l["flags"] & mtx.MTX_GEMM_FUSED_UPDATE]
    plain = [l for l in mtx.mtx_get_launches(b.handle) if l["flags"] & mtx.MTX_GEMM_FUSED_UPDATE]
    _say("[launches] fused: " + ", ".join(f"{l['site']}:L{l['layer']}:{l['tile_rows']}x"
                                          f"{l['tile_cols']}" for l in fused))
    assert sorted(l["layer"] for l in fused) == expect and not plain
    assert all(l["site"] == "wgrad_update" and l["splits"] == 1 for l in fused)
    a.close()
    b.close()


@pytest.mark.parametrize("name,R,Nb", [("lenet", 4, 8), ("alexnet", 2, 2)])
def test_nonfinite_check_is_bit_identical_when_finite(name, R, Nb):
    """With the non-finite check on, a step averages first, flags non-finite averages and then
    updates from the stored average: w, v, the average and the shard rows are bit-identical to
    the fused average + update (and, for AlexNet, to the fused fc updates) when all is finite."""
    net = {"lenet": wl.LENET, "alexnet": wl.ALEXNET}[name]
    layers = wl.layer_tuples(net)
    _say(f"[case] non-finite check, finite step {name} R={R} Nb={Nb}")
    a = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=8)
    b = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=8)
    mtx.mtx_set_nonfinite_check(a.handle, True)
    x, y = wl.make_batch(net, R * Nb, seed=8)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    for step in range(2):
        a.train_step(xd, yd, 0.01, 0.9)
        b.train_step(xd, yd, 0.01, 0.9)
        torch.cuda.synchronize()
        assert np.array_equal(a.grads_host().view(np.uint32), b.grads_host().view(np.uint32)), step
        wa, va = a.get_params()
        wb, vb = b.get_params()
        assert np.array_equal(wa.view(np.uint32), wb.view(np.uint32)), step
        assert np.array_equal(va.view(np.uint32), vb.view(np.uint32)), step
        ga, gb = a.grad_avg.cpu().numpy(), b.grad_avg.cpu().numpy()
        assert np.array_equal(ga.view(np.uint32), gb.view(np.uint32)), step
    a.close()
    b.close()


def test_nonfinite_check_skips_the_update():
    """An input with an infinite value makes the gradient average non-finite: the step returns
    MTX_ENONFINITE and leaves w and v as they were; the next finite step updates as usual.  The
    check refuses the adaptive update rules."""
    net = wl.LENET
    layers = wl.layer_tuples(net)
    R, Nb = 2, 4
    _say("[case] non-finite check, infinite input")
    m = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=9)
    mtx.mtx_set_nonfinite_check(m.handle, True)
    x, y = wl.make_batch(net, R * Nb, seed=9)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    m.train_step(xd, yd, 0.01, 0.9)  # finite: v becomes non-zero
    torch.cuda.synchronize()
    w0, v0 = m.get_params()
    assert np.any(v0 != 0)
    bad = x.copy()
    bad[1, 0, 3, 5] = np.inf
    with pytest.raises(mtx.MtxError) as err:
        m.train_step(torch.from_numpy(bad).cuda(), yd, 0.01, 0.9)
    assert err.value.code == mtx.MTX_ENONFINITE
    w1, v1 = m.get_params()
    assert np.array_equal(w1.view(np.uint32), w0.view(np.uint32))
    assert np.array_equal(v1.view(np.uint32), v0.view(np.uint32))
    assert not np.all(np.isfinite(m.grad_avg.cpu().numpy()))
    m.train_step(xd, yd, 0.01, 0.9)
    torch.cuda.synchronize()
    w2, _ = m.get_params()
    assert np.all(np.isfinite(w2)) and not np.array_equal(w2, w0)
    m.set_optimizer(mtx.MTX_OPT_ADAM, *ADAM)
    with pytest.raises(mtx.MtxError) as err:
        m.train_step(xd, yd, 1e-3, 0.0)
    assert err.value.code == mtx.MTX_EUNSUPPORTED
    m.close()


def _layerwise(model):
    mtx.mtx_set_overlap(model.handle, True)
    mtx.mtx_set_layerwise_update(model.handle, True)


@pytest.mark.parametrize("name,R,Nb", [("lenet", 4, 16), ("cifar", 8, 2), ("alexnet", 4, 1)])
def test_layerwise_update_step_matches_oracle(name, R, Nb):
    """Layer-wise average + update (Sec. III-D.2: one reduction per layer, in layer order; each
    layer's parameters averaged and updated on the third stream as soon as its R shard gradients
    are written, beside the rest of the backward pass, with the weight gradients on the second
    stream) against the oracle's step: gradients, average, velocity, update and every output."""
    net = {"lenet": wl.LENET, "cifar": wl.CIFAR, "alexnet": wl.ALEXNET}[name]
    run_case(f"{name}-layerwise", net, R, Nb, 2, 41, 0.01, 0.9, check_acts=name != "alexnet",
             configure=_layerwise)


def test_layerwise_update_on_one_stream_matches():
    """Layer-wise updates without the second stream (weight gradients on the caller's stream,
    each layer's update on the third) match the plain order bit for bit."""
    net = wl.LENET
    layers = wl.layer_tuples(net)
    _say("[case] layerwise update, one weight-gradient stream")
    a = mtx.Model(net.in_shape, layers, net.dtype, 4, 8, seed=5)
    b = mtx.Model(net.in_shape, layers, net.dtype, 4, 8, seed=5)
    mtx.mtx_set_overlap(a.handle, False)
    mtx.mtx_set_layerwise_update(a.handle, True)
    mtx.mtx_set_overlap(b.handle, False)
    x, y = wl.make_batch(net, 32, seed=5)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    for step in range(2):
        a.train_step(xd, yd, 0.01, 0.9)
        b.train_step(xd, yd, 0.01, 0.9)
        torch.cuda.synchronize()
        wa, va = a.get_params()
        wb, vb = b.get_params()
        assert np.array_equal(wa.view(np.uint32), wb.view(np.uint32)), step
        assert np.array_equal(va.view(np.uint32), vb.view(np.uint32)), step
        ga, gb = a.grad_avg.cpu().numpy(), b.grad_avg.cpu().numpy()
        assert np.array_equal(ga.view(np.uint32), gb.view(np.uint32)), step
    a.close()
    b.close()


@pytest.mark.parametrize("net_name", ["lenet", "cifar"])
def test_shard_count_invariance(net_name):
    """Synchronous SGD does not depend on how the batch is split (Sec. III-E): three steps on
    the same batches with R = 1, 2, 4, 8 shards give the same weight change up to rounding (the
    averages of shard means are summed in another order)."""
    net = {"lenet": wl.LENET, "cifar": wl.CIFAR}[net_name]
    layers = wl.layer_tuples(net)
    B = 16
    tol = parity.TOL[net.dtype]
    _say(f"[case] shard-count invariance {net_name}")
    deltas = {}
    for R in (1, 2, 4, 8):
        m = mtx.Model(net.in_shape, layers, net.dtype, R, B // R, seed=11)
        w0, _ = m.get_params()
        for step in range(3):
            x, y = wl.make_batch(net, B, seed=100 + step)
            m.train_step(torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), 0.01, 0.9)
        torch.cuda.synchronize()
        w3, _ = m.get_params()
        deltas[R] = w3.astype(np.float64) - w0.astype(np.float64)
        m.close()
    ref = deltas[1]
    for R in (2, 4, 8):
        d = deltas[R]
        assert np.linalg.norm(d - ref) <= tol * np.linalg.norm(ref), R
        assert np.max(np.abs(d - ref)) <= tol * np.max(np.abs(ref)) + 1e-7, R


@pytest.mark.parametrize("net_name,R,Nb,steps,lr,mu", [("mlp", 2, 32, 10, 0.01, 0.0),
                                                        ("lenet", 4, 8, 10, 0.01, 0.9),
                                                        ("lenet", 1, 32, 10, 0.01, 0.9)])
def test_free_running_trajectory_matches_oracle(net_name, R, Nb, steps, lr, mu):
    """Several steps with no state copied between the two sides (the analogue of the paper's
    loss curves, Fig. 7): the GPU model and the oracle each start from the same initial weights
    and run `steps` steps on the same batches from their own state.  The per-step losses and
    the total weight change must agree to the parity tolerance; with fp32 compute the rounding
    differences that accumulate over the steps stay well inside it.  (bf16 steps are compared
    from a shared state each step, in the tests above: once two bf16 trajectories differ by
    rounding, ReLU and pooling decisions near ties flip, which no per-step hint can follow; over
    four CIFAR steps that moved the total weight change by 8% with the losses still agreeing to
    2e-2.)"""
    net = {"mlp": wl.MLP, "lenet": wl.LENET}[net_name]
    layers = wl.layer_tuples(net)
    prec = "f32"
    tol = parity.TOL[net.dtype]
    _say(f"[case] free-running trajectory {net_name} R={R} Nb={Nb} steps={steps}")
    model = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=21)
    w0 = orc.init_glorot(net.in_shape, layers, 21)
    w, v = w0.copy(), np.zeros_like(w0)
    loss_dev = torch.zeros(1, device="cuda")
    lg, lo = [], []
    for step in range(steps):
        x, y = wl.make_batch(net, R * Nb, seed=5000 + step)
        model.train_step(torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), lr, mu, loss_dev)
        res = orc.train_step(net.in_shape, layers, R, x, y, w, v if mu else None, lr, mu,
                             prec=prec, want_grads=False)
        lg.append(float(loss_dev.item()))
        lo.append(res.loss)
        w = res.w_new
        if mu:
            v = res.v_new
    torch.cuda.synchronize()
    wg, vg = model.get_params()
    model.close()
    lg, lo = np.array(lg), np.array(lo)
    assert np.all(np.abs(lg - lo) <= tol * np.abs(lo)), (lg, lo)
    parity.assert_update_close(wg, w, w0, tol, "w after the trajectory")
    if mu:
        parity.assert_tensor_close(vg, v, tol, "velocity after the trajectory")
    # the trajectory went somewhere: the loss moved over the steps
    assert abs(lo[-1] - lo[0]) > 10 * tol * abs(lo[0])


# ---- Adam and AdaGrad as the update rule of the training step ----------------------------------

ADAM = (0.9, 0.999, 1e-8)


@pytest.mark.parametrize("kind", [mtx.MTX_OPT_ADAM, mtx.MTX_OPT_ADAGRAD])
@pytest.mark.parametrize("layerwise", [False, True])
def test_train_step_with_adaptive_update_equals_gradients_then_update(kind, layerwise):
    """A step with Adam / AdaGrad selected is bit-identical to a step that only computes the
    gradients (lr = 0, no momentum) followed by mtx_adam_update / mtx_adagrad_update on them
    (whose arithmetic the update tests compare with the oracle), over three steps; also with the
    per-layer update on the third stream."""
    net = wl.LENET
    layers = wl.layer_tuples(net)
    R, Nb, lr = 4, 8, 1e-3
    _say(f"[case] adaptive update in the step kind={kind} layerwise={layerwise}")
    a = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=3)
    b = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=3)
    a.set_optimizer(kind, *ADAM)
    w_init, _ = a.get_params()
    if layerwise:
        mtx.mtx_set_overlap(a.handle, True)
        mtx.mtx_set_layerwise_update(a.handle, True)
    if kind == mtx.MTX_OPT_ADAGRAD:
        w0, _ = a.get_params()
        acc0 = wl.make_square_state(a.P, seed=3, terms=2)
        a.set_params(w0, acc0)
        b.set_params(w0, acc0)
    s2b = torch.zeros(b.P, device="cuda")
    avg_b = torch.empty(b.P, device="cuda")
    for t in (1, 2, 3):
        x, y = wl.make_batch(net, R * Nb, seed=70 + t)
        xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
        a.train_step(xd, yd, lr, 0.0)
        b.train_step(xd, yd, 0.0, 0.0)
        if kind == mtx.MTX_OPT_ADAM:
            mtx.mtx_adam_update(b.w, b.v, s2b, b.grads, R, b.P, b.ld, lr, *ADAM, t, avg_b)
        else:
            mtx.mtx_adagrad_update(b.w, b.v, b.grads, R, b.P, b.ld, lr, ADAM[2], avg_b)
        torch.cuda.synchronize()
        wa, va = a.get_params()
        wb, vb = b.get_params()
        assert np.array_equal(wa.view(np.uint32), wb.view(np.uint32)), t
        assert np.array_equal(va.view(np.uint32), vb.view(np.uint32)), t
        assert torch.equal(a.grad_avg, avg_b), t
        if kind == mtx.MTX_OPT_ADAM:
            assert torch.equal(a.s2, s2b), t
    assert np.abs(wa - w_init).max() > 0  # the steps moved the weights
    a.close()
    b.close()


@pytest.mark.parametrize("kind", [mtx.MTX_OPT_ADAM, mtx.MTX_OPT_ADAGRAD])
def test_train_step_with_adaptive_update_matches_oracle(kind):
    """Three steps of LeNet (B = 32, R = 4) with Adam / AdaGrad inside mtx_train_step against the
    oracle's step gradients followed by its Adam / AdaGrad, each step from the same state.  The
    incoming second moment (Adam) and accumulator (AdaGrad) are non-zero, so the update is
    well-conditioned and the gradients' own rounding differences stay within tolerance."""
    net = wl.LENET
    layers = wl.layer_tuples(net)
    geo = orc.geometry(net.in_shape, layers)
    R, Nb, lr = 4, 8, 1e-3
    tol = parity.TOL[net.dtype]
    _say(f"[case] adaptive update vs oracle kind={kind}")
    model = mtx.Model(net.in_shape, layers, net.dtype, R, Nb, seed=8)
    model.set_optimizer(kind, *ADAM)
    P = model.P
    w = orc.init_glorot(net.in_shape, layers, 8)
    s1 = wl.make_velocity(P, seed=8) if kind == mtx.MTX_OPT_ADAM else wl.make_square_state(P, seed=8, terms=4)
    s2 = wl.make_square_state(P, seed=9, terms=4)
    for t in (1, 2, 3):
        x, y = wl.make_batch(net, R * Nb, seed=90 + t)
        model.set_params(w, s1)
        if kind == mtx.MTX_OPT_ADAM:
            model.s2.copy_(torch.from_numpy(s2).cuda())
        model.train_step(torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), lr, 0.0)
        torch.cuda.synchronize()
        gp, gr = parity.gpu_decisions(model, geo)
        res, _ = parity.oracle_step_matching(net, layers, R, x, y, w, None, 0.0, 0.0, "f32", gp, gr)
        if kind == mtx.MTX_OPT_ADAM:
            gavg, w_new, s1_new, s2_new = orc.average_adam(res.grads, w, s1, s2, lr, *ADAM, t)
        else:
            gavg, w_new, s1_new = orc.average_adagrad(res.grads, w, s1, lr, ADAM[2])
        wg, s1g = model.get_params()
        parity.assert_tensor_close(model.grad_avg.cpu().numpy(), gavg, tol, f"average t={t}")
        parity.assert_tensor_close(s1g, s1_new, tol, f"first state t={t}")
        parity.assert_update_close(wg, w_new, w, tol, f"w t={t}")
        if kind == mtx.MTX_OPT_ADAM:
            parity.assert_tensor_close(model.s2.cpu().numpy(), s2_new, tol, f"second moment t={t}")
            s2 = s2_new
        w, s1 = w_new, s1_new
    model.close()


# ---- batch normalisation and residual additions (Table II's ResNet-50 building blocks) ---------

@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_residual_batchnorm_network(dtype):
    run_case("residual-bn", _residual(dtype), 3, 4, 2, seed=31, lr=0.01, mu=0.9)


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_residual_batchnorm_edge_layers(dtype):
    run_case("residual-edges", _residual_edges(dtype), 2, 5, 2, seed=32, lr=0.01, mu=0.9)


def _projection(dtype):
    """A downsampling block with a projection shortcut (strided 1x1 convolution of layer 1's
    output added to the strided main path), an identity block, and a stride-1 projection whose
    source has no ReLU, then pooling and the classifier."""
    layers = (wl.conv(8, 3, pad=1), wl.bn(relu=True),
              wl.conv(16, 3, stride=2, pad=1), wl.bn(), wl.addp(1, 16, stride=2, relu=True),
              wl.conv(16, 3, pad=1), wl.bn(), wl.add(4, relu=True),
              wl.conv(24, 1), wl.addp(6, 24), wl.maxpool(2, 2), wl.fc(5))
    return wl.Net("projection", (3, 12, 12), layers, dtype, "normal")


@pytest.mark.parametrize("dtype", [wl.F32, wl.BF16])
def test_projection_shortcut_network(dtype):
    run_case(f"projection-{dtype}", _projection(dtype), 2, 4, 2, seed=35, lr=0.01, mu=0.9)


def test_bottleneck_shapes_fp32_reduced_batch():
    """The bottleneck workload's layer shapes (1x1-3x3-1x1 blocks, projection shortcuts, a
    stride-2 downsampling block) with fp32 compute at B = 4, R = 2, to the fp32 bound."""
    net = wl.Net("bottleneck-f32", wl.RESNET_BOTTLENECK.in_shape, wl.RESNET_BOTTLENECK.layers,
                 wl.F32, "normal")
    run_case("bottleneck fp32", net, 2, 2, 1, seed=36, lr=0.01, mu=0.9)


def test_bottleneck_workload_reduced_batch():
    run_case("bottleneck", wl.RESNET_BOTTLENECK, 2, 16, 1, seed=37, lr=0.01, mu=0.9,
             tol=parity.RESNET_TOL)


def test_resnet_shapes_fp32_reduced_batch():
    """The residual workload's exact layer shapes with fp32 compute at B = 4, R = 2, to the fp32
    bound: every kernel of the 30-layer network (measured: about 1e-6 at every layer)."""
    net = wl.Net("resnet-f32", wl.RESNET.in_shape, wl.RESNET.layers, wl.F32, "normal")
    run_case("resnet fp32", net, 2, 2, 1, seed=33, lr=0.01, mu=0.9)


def test_resnet_workload_reduced_batch():
    """The residual workload itself (bf16) at B = 32, R = 2.  Its 28 bf16-stored activations and
    data gradients in sequence, with per-shard batch normalisation, let any two fp32 evaluations
    drift apart with depth: an independent fp32 evaluation on the CPU lies 1.7e-2 from the oracle
    with 16 samples per shard, about 3e-2 with 4 (test_oracle_spread.py) and up to 2.2e-2 with
    64.  The bound is parity.RESNET_TOL = 3e-2 (2e-2 is not attainable for this network),
    and the reduced batch keeps 16 samples per shard."""
    run_case("resnet", wl.RESNET, 2, 16, 1, seed=33, lr=0.01, mu=0.9, tol=parity.RESNET_TOL)


def test_resnet_full_batch_runs_and_shards_are_independent():
    """The residual workload at its full size (B = 512, R = 8) in the launch configuration the
    benchmark times: finite loss and gradients, and every shard's gradient row differs (each
    shard is normalised by its own statistics and sees its own samples)."""
    w = wl.WORKLOADS["resnet"]
    net = w.net
    _say("[case] resnet full size")
    model = mtx.Model(net.in_shape, wl.layer_tuples(net), net.dtype, w.shards, w.shard_batch,
                      seed=0)
    x, y = wl.make_batch(net, w.batch, seed=0)
    loss = torch.zeros(1, device="cuda")
    model.train_step(torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), w.lr, w.momentum,
                     loss)
    torch.cuda.synchronize()
    g = model.grads_host()
    assert np.isfinite(float(loss.item())) and np.all(np.isfinite(g))
    avg = model.grad_avg.cpu().numpy()
    assert np.allclose(avg, g.astype(np.float64).mean(0), rtol=1e-5, atol=1e-7 * np.abs(avg).max())
    for r in range(1, w.shards):
        assert not np.array_equal(g[0], g[r])
    model.close()
