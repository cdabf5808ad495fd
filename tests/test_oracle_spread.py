"""How far two legitimate evaluations of a bf16 step can lie apart.  CPU only.

The GPU sums in fp32 (in its own order) between the bf16 rounding points; the oracle sums in
fp64.  An independent evaluation of the same kind as the GPU's -- torch on the CPU in float32,
with the same bf16 storage points (tests/torch_ref.fp32_evaluation_bf16) -- shows how far such
an evaluation lies from the oracle when its pooling and ReLU decisions are handed to the oracle
exactly as the GPU's are.  For the eleven-layer CIFAR network this is far inside the 2e-2 bound.
For the 30-layer residual network with per-shard batch normalisation it is not: each BN layer
divides by the shard's standard deviation, and 28 bf16 roundings of activations and data
gradients lie in sequence.  With 4 samples per shard the spread is about 3e-2; with 16 it is
about 1.7e-2; with the benchmark's 64 it was measured at 1.6e-2 to 2.2e-2 over three seeds (the
largest on the shift gradient of a batch normalisation layer).  The 2e-2 bound is therefore not
attainable for this network by any fp32 evaluation, the GPU's included; its GPU tests use 3e-2
and shards of at least 16 samples.
"""
import numpy as np
import pytest

from oracle import oracle as orc
from paper_1704_04560_amd import workloads as wl
from tests import parity, torch_ref


def _spread(net, Nb, seed):
    layers = wl.layer_tuples(net)
    geo = orc.geometry(net.in_shape, layers)
    w = orc.init_glorot(net.in_shape, layers, seed)
    x, y = wl.make_batch(net, Nb, seed=seed)
    g, acts, gp, gr = torch_ref.fp32_evaluation_bf16(layers, geo, w, x, y)
    res, _ = parity.oracle_step_matching(net, layers, 1, x, y, w, None, 0.0, 0.0, "bf16", gp, gr,
                                         tag=f"{net.name} fp32 evaluation Nb={Nb}")
    worst_grad = max(max(parity.rel_err(g[gg["w_off"]:gg["w_off"] + gg["w_len"]],
                                        res.grads[0][gg["w_off"]:gg["w_off"] + gg["w_len"]]))
                     for gg in geo if gg["w_len"])
    off, worst_out = 0, 0.0
    for gi, gg in enumerate(geo):
        n = acts[gi].size
        worst_out = max(worst_out, max(parity.rel_err(acts[gi], res.acts[off:off + n])))
        off += n
    return worst_grad, worst_out


def test_cifar_fp32_evaluation_is_far_inside_the_bound():
    wg, wo = _spread(wl.CIFAR, 8, 5)
    assert wg < 5e-3 and wo < 1e-2, (wg, wo)


def test_residual_network_spread_exceeds_the_bound_with_four_samples_per_shard():
    wg, wo = _spread(wl.RESNET, 4, 5)
    assert wg > 2e-2, (wg, wo)


@pytest.mark.slow
def test_residual_network_spread_with_sixteen_samples_per_shard():
    wg, wo = _spread(wl.RESNET, 16, 5)
    assert wg <= parity.RESNET_TOL and wo <= parity.RESNET_TOL, (wg, wo)
