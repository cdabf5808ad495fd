"""Seeded synthetic workloads shaped like the paper's training runs.

This module holds data only: network descriptions and seeded input generators.  It contains
none of the method's arithmetic and imports nothing from the GPU library or from the oracle, so
both sides (and the tests and the benchmark) can draw identical inputs from it.

Networks (the paper evaluates MLP/CNN image classifiers, Sec. I and Fig. 1, with ImageNet-sized
AlexNet as its hardest case to scale, Sec. IV; no dataset is read, the inputs are seeded random
tensors of the same shapes):
  mlp      784-256-10 MLP, ReLU, fp32, B=64 split into R=2 shards, plain SGD lr=0.01
  lenet    LeNet-style CNN fp32, [256,1,28,28] U(0,1), R=4, momentum 0.9, lr=0.01
  cifar    CIFAR-style CNN, bf16 compute, [512,3,32,32] N(0,1), R=8, momentum 0.9, lr=0.01
  alexnet  AlexNet-shaped CNN (groups=2 on conv2/4/5), bf16 compute, [256,3,227,227] N(0,1),
           1000 classes, R=8, momentum 0.9, lr=0.01
  resnet   residual CNN with batch normalisation (the building blocks of Table II's ResNet-50
           at CIFAR scale), bf16 compute, [512,3,32,32] N(0,1), R=8, momentum 0.9, lr=0.01
Gradient-average microbenchmark: R=16 buffers of n elements, N(0, 1e-3) gradients, N(0, 0.05)
weights, N(0, 1e-3) velocity, momentum 0.9, lr 0.01.

Random streams: numpy.random.default_rng([seed, stream]) with stream 0 = input images,
1 = labels, 2 = weights (when a test draws its own), 3 = velocity, 4 = gradient buffers,
5 = second optimizer state (Adam's second moment, AdaGrad's accumulator).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np

FC, CONV, MAXPOOL, BN, ADD, ADDP = 0, 1, 2, 3, 4, 5
F32, BF16 = 0, 1

STREAM_X, STREAM_LABELS, STREAM_W, STREAM_V, STREAM_G, STREAM_S2 = 0, 1, 2, 3, 4, 5


@dataclass(frozen=True)
class Layer:
    kind: int
    out: int = 0
    k: int = 1
    stride: int = 1
    pad: int = 0
    groups: int = 1
    relu: bool = False


def fc(out, relu=False):
    return Layer(FC, out, 1, 1, 0, 1, relu)


def conv(out, k, stride=1, pad=0, groups=1, relu=False):
    return Layer(CONV, out, k, stride, pad, groups, relu)


def maxpool(k, stride):
    return Layer(MAXPOOL, 0, k, stride, 0, 1, False)


def bn(relu=False):
    """Batch normalisation over the shard, gamma and beta per channel."""
    return Layer(BN, 0, 0, 1, 0, 1, relu)


def add(src, relu=False):
    """Residual addition of the output of layer `src` (an earlier layer of the same shape)."""
    return Layer(ADD, 0, src, 1, 0, 1, relu)


def addp(src, out, stride=1, relu=False):
    """Residual addition through a projection shortcut: the output of layer `src` passes a 1x1
    convolution of the given stride (out = this layer's channel count, with weights and bias)
    and is added to the previous layer's output (ResNet-50's downsampling blocks)."""
    return Layer(ADDP, out, src, stride, 0, 1, relu)


@dataclass(frozen=True)
class Net:
    name: str
    in_shape: Tuple[int, int, int]  # (C, H, W) per sample
    layers: Tuple[Layer, ...]
    dtype: int  # F32 or BF16 compute
    x_dist: str  # "normal" or "uniform"

    @property
    def num_classes(self) -> int:
        return self.layers[-1].out


@dataclass(frozen=True)
class Workload:
    net: Net
    batch: int
    shards: int
    lr: float
    momentum: float
    description: str = field(default="")

    @property
    def shard_batch(self) -> int:
        return self.batch // self.shards


MLP = Net("mlp", (784, 1, 1), (fc(256, relu=True), fc(10)), F32, "normal")

# LeNet as the workload describes it: the two convolutions carry no ReLU.
LENET = Net("lenet", (1, 28, 28),
            (conv(20, 5), maxpool(2, 2), conv(50, 5), maxpool(2, 2), fc(500, relu=True), fc(10)),
            F32, "uniform")

CIFAR = Net("cifar", (3, 32, 32),
            (conv(64, 3, pad=1, relu=True), conv(64, 3, pad=1, relu=True), maxpool(2, 2),
             conv(128, 3, pad=1, relu=True), conv(128, 3, pad=1, relu=True), maxpool(2, 2),
             conv(256, 3, pad=1, relu=True), conv(256, 3, pad=1, relu=True), maxpool(2, 2),
             fc(10)),
            BF16, "normal")

# AlexNet in the two-group layout of the original network (conv2, conv4, conv5 split in two
# groups); no local response normalisation and no dropout.  60,965,224 parameters.
ALEXNET = Net("alexnet", (3, 227, 227),
              (conv(96, 11, stride=4, relu=True), maxpool(3, 2),
               conv(256, 5, pad=2, groups=2, relu=True), maxpool(3, 2),
               conv(384, 3, pad=1, relu=True),
               conv(384, 3, pad=1, groups=2, relu=True),
               conv(256, 3, pad=1, groups=2, relu=True), maxpool(3, 2),
               fc(4096, relu=True), fc(4096, relu=True), fc(1000)),
              BF16, "normal")

# A residual network in the manner of Table II's ResNet-50 at CIFAR scale: 3x3 convolutions,
# batch normalisation (per-shard statistics), identity shortcuts around pairs of convolutions,
# 2/2 max-pooling between the three widths (64, 128, 256), a fully connected classifier.
def _res_block(first, width):
    """conv-BN-ReLU-conv-BN, added to the output of layer `first` - 1, then ReLU."""
    return (conv(width, 3, pad=1), bn(relu=True), conv(width, 3, pad=1), bn(),
            add(first - 1, relu=True))


# ResNet-50's bottleneck blocks at CIFAR scale: 1x1 - 3x3 - 1x1 convolutions with batch
# normalisation, identity shortcuts within a stage and projection shortcuts (strided 1x1
# convolutions) where a block changes width or resolution; the 3x3 convolution of a downsampling
# block has stride 2.
def _bottleneck(first, width, out, src, stride=1, proj=False):
    """Layers first .. first+6: conv1x1-BN-ReLU, conv3x3(stride)-BN-ReLU, conv1x1-BN, shortcut
    from layer src (projection or identity), ReLU."""
    return (conv(width, 1), bn(relu=True), conv(width, 3, stride=stride, pad=1), bn(relu=True),
            conv(out, 1), bn(),
            addp(src, out, stride=stride, relu=True) if proj else add(src, relu=True))


RESNET_BOTTLENECK = Net("resnet-bottleneck", (3, 32, 32),
                        (conv(64, 3, pad=1), bn(relu=True))                  # 0-1
                        + _bottleneck(2, 64, 256, 1, proj=True)              # 2-8
                        + _bottleneck(9, 64, 256, 8)                         # 9-15
                        + _bottleneck(16, 128, 512, 15, stride=2, proj=True)  # 16-22, 16x16
                        + _bottleneck(23, 128, 512, 22)                      # 23-29
                        + (maxpool(4, 4), fc(10)),                           # 30-31
                        BF16, "normal")

RESNET = Net("resnet", (3, 32, 32),
             (conv(64, 3, pad=1), bn(relu=True))                      # 0-1
             + _res_block(2, 64) + _res_block(7, 64) + (maxpool(2, 2),)  # 2-12
             + (conv(128, 3, pad=1), bn(relu=True))                   # 13-14
             + _res_block(15, 128) + (maxpool(2, 2),)                 # 15-20
             + (conv(256, 3, pad=1), bn(relu=True))                   # 21-22
             + _res_block(23, 256) + (maxpool(2, 2), fc(10)),         # 23-29
             BF16, "normal")

WORKLOADS = {
    "mlp": Workload(MLP, 64, 2, 0.01, 0.0, "MLP 784-256-10 fp32, B=64, R=2, SGD"),
    "lenet": Workload(LENET, 256, 4, 0.01, 0.9, "LeNet fp32, B=256, R=4, momentum 0.9"),
    "cifar": Workload(CIFAR, 512, 8, 0.01, 0.9, "CIFAR CNN bf16, B=512, R=8, momentum 0.9"),
    "alexnet": Workload(ALEXNET, 256, 8, 0.01, 0.9, "AlexNet bf16, B=256, R=8, momentum 0.9"),
    "resnet": Workload(RESNET, 512, 8, 0.01, 0.9,
                       "residual CNN with batch norm bf16, B=512, R=8, momentum 0.9"),
    "bottleneck": Workload(RESNET_BOTTLENECK, 256, 8, 0.01, 0.9,
                           "bottleneck residual CNN with projection shortcuts bf16, B=256, R=8, "
                           "momentum 0.9"),
}

AVG_UPDATE = {"R": 16, "n": (61_000_000, 250_000_000), "lr": 0.01, "momentum": 0.9,
              "grad_std": 1e-3, "w_std": 0.05, "v_std": 1e-3}


def rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(stream)])


def make_batch(net: Net, batch: int, seed: int = 0):
    """Input images [batch, C, H, W] float32 and labels [batch] int32."""
    c, h, w = net.in_shape
    g = rng(seed, STREAM_X)
    if net.x_dist == "uniform":
        x = g.random((batch, c, h, w), dtype=np.float32)
    else:
        x = g.standard_normal((batch, c, h, w), dtype=np.float32)
    y = rng(seed, STREAM_LABELS).integers(0, net.num_classes, size=batch, dtype=np.int32)
    return x, y


def make_params(n_params: int, seed: int = 0, scale: float = 0.05) -> np.ndarray:
    """Random parameter vector (used where a test sets parameters instead of the library's
    own initialisation)."""
    return (rng(seed, STREAM_W).standard_normal(n_params, dtype=np.float32) * np.float32(scale))


def make_velocity(n_params: int, seed: int = 0, scale: float = 1e-3) -> np.ndarray:
    return (rng(seed, STREAM_V).standard_normal(n_params, dtype=np.float32) * np.float32(scale))


def make_avg_update_inputs(R: int, n: int, seed: int = 0, ld: int | None = None):
    """Host inputs of the gradient-average microbenchmark: grads [R][ld] (only the first n of
    each row are drawn; the rest are zero), w [n], v [n]."""
    ld = n if ld is None else ld
    spec = AVG_UPDATE
    grads = np.zeros((R, ld), dtype=np.float32)
    grads[:, :n] = rng(seed, STREAM_G).normal(0.0, spec["grad_std"], size=(R, n)).astype(np.float32)
    w = rng(seed, STREAM_W).normal(0.0, spec["w_std"], size=n).astype(np.float32)
    v = rng(seed, STREAM_V).normal(0.0, spec["v_std"], size=n).astype(np.float32)
    return grads, w, v


def make_square_state(n: int, seed: int = 0, terms: int = 1) -> np.ndarray:
    """Non-negative state of the size a running sum or average of squared gradients takes:
    the sum of `terms` squares of N(0, 1e-3) draws, as float32 [n]."""
    z = rng(seed, STREAM_S2).normal(0.0, AVG_UPDATE["grad_std"], size=(terms, n))
    return (z * z).sum(axis=0).astype(np.float32)


def layer_tuples(net: Net) -> List[Tuple[int, int, int, int, int, int, int]]:
    return [(l.kind, l.out, l.k, l.stride, l.pad, l.groups, int(l.relu)) for l in net.layers]
