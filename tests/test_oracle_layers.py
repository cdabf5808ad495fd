"""Pins of the oracle's single layers against torch float64 autograd (an independent
implementation of the same textbook definitions).  CPU only."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import oracle as orc

RTOL = 1e-11


def _close(a, b, rtol=RTOL):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    scale = max(1.0, float(np.max(np.abs(b))) if b.size else 1.0)
    assert a.shape == b.shape
    assert np.max(np.abs(a - b)) <= rtol * scale, np.max(np.abs(a - b))


CONV_CASES = [
    # N, C, H, W, OC, K, S, P, G
    (2, 1, 9, 9, 4, 5, 1, 0, 1),      # LeNet-like 5x5 valid
    (2, 3, 8, 8, 6, 3, 1, 1, 1),      # CIFAR-like 3x3 same
    (1, 3, 23, 23, 4, 11, 4, 0, 1),   # AlexNet conv1-like 11x11 stride 4
    (2, 4, 7, 7, 6, 5, 1, 2, 2),      # grouped 5x5 pad 2
    (1, 6, 5, 6, 4, 3, 2, 1, 2),      # grouped, stride 2, non-square
    (3, 2, 4, 4, 3, 1, 1, 0, 1),      # 1x1
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_matches_torch(case):
    N, Cc, H, W, OC, K, S, P, G = case
    g = np.random.default_rng(list(case))
    x = g.standard_normal((N, Cc, H, W))
    w = g.standard_normal((OC, Cc // G, K, K))
    b = g.standard_normal(OC)
    y = orc.conv_fwd(x, w, b, S, P, G)
    xt = torch.tensor(x, requires_grad=True)
    wt = torch.tensor(w, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    yt = F.conv2d(xt, wt, bt, stride=S, padding=P, groups=G)
    _close(y, yt.detach().numpy())
    dy = g.standard_normal(y.shape)
    yt.backward(torch.tensor(dy))
    dx, dw, db = orc.conv_bwd(x, w, dy, S, P, G)
    _close(dx, xt.grad.numpy())
    _close(dw, wt.grad.numpy())
    _close(db, bt.grad.numpy())


@pytest.mark.parametrize("N,IN,OUT", [(3, 7, 5), (1, 1, 1), (4, 33, 2)])
def test_fc_matches_torch(N, IN, OUT):
    g = np.random.default_rng([N, IN, OUT])
    x = g.standard_normal((N, IN))
    w = g.standard_normal((OUT, IN))
    b = g.standard_normal(OUT)
    y = orc.fc_fwd(x, w, b)
    xt = torch.tensor(x, requires_grad=True)
    wt = torch.tensor(w, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    yt = F.linear(xt, wt, bt)
    _close(y, yt.detach().numpy())
    dy = g.standard_normal(y.shape)
    yt.backward(torch.tensor(dy))
    dx, dw, db = orc.fc_bwd(x, w, dy)
    _close(dx, xt.grad.numpy())
    _close(dw, wt.grad.numpy())
    _close(db, bt.grad.numpy())


@pytest.mark.parametrize("N,C,H,W,K,S", [(2, 3, 8, 8, 2, 2), (2, 2, 11, 11, 3, 2),
                                         (1, 1, 7, 9, 3, 2), (1, 2, 5, 5, 2, 1)])
def test_maxpool_matches_torch(N, C, H, W, K, S):
    g = np.random.default_rng([N, C, H, W, K, S])
    x = g.standard_normal((N, C, H, W))
    y, am = orc.maxpool_fwd(x, K, S)
    xt = torch.tensor(x, requires_grad=True)
    yt = F.max_pool2d(xt, K, S)
    _close(y, yt.detach().numpy(), 0.0)
    dy = g.standard_normal(y.shape)
    yt.backward(torch.tensor(dy))
    dx = orc.maxpool_bwd(x.shape, K, S, am, dy)
    _close(dx, xt.grad.numpy())


def test_maxpool_tie_takes_first_in_row_major_order():
    x = np.zeros((1, 1, 2, 2))
    x[0, 0] = [[1.0, 3.0], [3.0, 2.0]]
    y, am = orc.maxpool_fwd(x, 2, 2)
    assert y[0, 0, 0, 0] == 3.0 and am[0, 0, 0, 0] == 1
    x[0, 0] = [[5.0, 5.0], [5.0, 5.0]]
    _, am = orc.maxpool_fwd(x, 2, 2)
    assert am[0, 0, 0, 0] == 0


@pytest.mark.parametrize("N,NC", [(4, 10), (3, 1000), (1, 2)])
def test_softmax_xent_matches_torch(N, NC):
    g = np.random.default_rng([N, NC])
    z = g.standard_normal((N, NC)) * 3
    y = g.integers(0, NC, size=N).astype(np.int32)
    loss, dz = orc.softmax_xent(z, y, 1.0 / N)
    zt = torch.tensor(z, requires_grad=True)
    lt = F.cross_entropy(zt, torch.tensor(y, dtype=torch.long), reduction="none")
    _close(loss, lt.detach().numpy())
    lt.mean().backward()
    _close(dz, zt.grad.numpy())


def test_softmax_xent_zero_logits_give_log_c_exactly():
    for NC in (10, 1000):
        z = np.zeros((3, NC))
        loss, dz = orc.softmax_xent(z, np.array([0, 5, NC - 1], dtype=np.int32), 1.0 / 3)
        assert np.all(loss == np.log(NC))
        assert np.allclose(dz.sum(axis=1), 0.0, atol=1e-15)


def test_softmax_xent_large_logits_are_stable():
    z = np.array([[1000.0, 0.0, -1000.0]])
    loss, dz = orc.softmax_xent(z, np.array([0], dtype=np.int32), 1.0)
    assert loss[0] == 0.0 and np.all(np.isfinite(dz))
