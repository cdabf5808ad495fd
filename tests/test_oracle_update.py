"""Pins of the oracle's average + momentum update, weight initialisation and bfloat16 rounding.
CPU only."""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_1704_04560_amd import workloads as wl


@pytest.mark.parametrize("mu", [0.0, 0.9, 0.5])
def test_momentum_closed_form_for_constant_gradient(mu):
    """With a constant gradient g and v0 = 0: v_k = g (1 - mu^k) / (1 - mu) and
    w_k = w_0 - lr g sum_{j=1..k} (1 - mu^j) / (1 - mu) (mu = 0 reduces to plain SGD)."""
    n, R, lr, steps = 257, 4, 0.01, 6
    rng = np.random.default_rng(0)
    g = rng.normal(0, 1e-2, n)
    # R identical rows whose values have few significant bits average exactly
    g = np.round(g * 2 ** 12) / 2 ** 12
    grads = np.tile(g.astype(np.float32), (R, 1))
    w0 = rng.normal(0, 1, n).astype(np.float32)
    w, v = w0.copy(), (np.zeros(n, np.float32) if mu else None)
    for _ in range(steps):
        gavg, w, v = orc.average_update(grads, w, v, lr, mu)
        assert np.array_equal(gavg, g.astype(np.float32))
    if mu:
        vk = g * (1 - mu ** steps) / (1 - mu)
        assert np.allclose(v, vk, rtol=1e-6, atol=1e-9)
        wk = w0 - lr * g * sum((1 - mu ** j) / (1 - mu) for j in range(1, steps + 1))
    else:
        wk = w0 - lr * g * steps
    assert np.allclose(w, wk, rtol=0, atol=steps * 2e-7)


def test_average_of_distinct_rows_and_row_stride():
    R, n, ld = 3, 10, 16
    grads = np.zeros((R, ld), np.float32)
    grads[:, :n] = np.arange(R * n, dtype=np.float32).reshape(R, n)
    grads[:, n:] = 1e9  # padding beyond n must not be read
    gavg, _, _ = orc.average_update(grads, np.zeros(n, np.float32), None, 0.1, 0.0, n=n)
    assert np.array_equal(gavg, np.arange(n, dtype=np.float32) + n)


def test_first_momentum_step_from_zero_velocity_equals_plain_sgd():
    grads, w, _ = wl.make_avg_update_inputs(4, 1001, seed=3)
    _, w_sgd, _ = orc.average_update(grads, w, None, 0.01, 0.0)
    _, w_mom, v_mom = orc.average_update(grads, w, np.zeros_like(w), 0.01, 0.9)
    assert np.array_equal(w_sgd, w_mom)


def test_glorot_init_range_moments_and_determinism():
    net = wl.LENET
    layers = wl.layer_tuples(net)
    geo = orc.geometry(net.in_shape, layers)
    w = orc.init_glorot(net.in_shape, layers, seed=123)
    assert np.array_equal(w, orc.init_glorot(net.in_shape, layers, seed=123))
    assert not np.array_equal(w, orc.init_glorot(net.in_shape, layers, seed=124))
    for g in geo:
        if g["kind"] == 2:
            continue
        c, h, ww = g["in_shape"]
        oc = g["out_shape"][0]
        if g["kind"] == 1:
            k = int(round((g["w_len"] / (oc * c)) ** 0.5))
            fan_in, fan_out = c * k * k, oc * k * k
        else:
            fan_in, fan_out = c * h * ww, oc
        a = np.sqrt(6.0 / (fan_in + fan_out))
        W = w[g["w_off"]:g["w_off"] + g["w_len"]].astype(np.float64)
        assert np.all(W >= -a) and np.all(W < a)
        assert abs(W.mean()) < 4 * a / np.sqrt(3 * W.size)
        assert abs(W.var() / (a * a / 3) - 1) < 6 * np.sqrt(0.8 / W.size) + 1e-3
        assert np.all(w[g["b_off"]:g["b_off"] + g["b_len"]] == 0)


def test_bf16_rounding_matches_torch_and_ties_to_even():
    cases = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -7, -(1 + 2 ** -8), 3.0e38,
                      1e-40, 0.0, -0.0, np.inf, -np.inf], dtype=np.float32)
    ours = orc.round_bf16(cases)
    assert ours[1] == 1.0                    # tie -> even (down)
    assert ours[2] == 1 + 2 ** -6            # tie -> even (up)
    assert ours[3] == 1 + 2 ** -7            # representable
    ref = torch.tensor(cases).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))
    r = np.random.default_rng(0).standard_normal(2000).astype(np.float32) * 1e3
    assert np.array_equal(orc.round_bf16(r), torch.tensor(r).to(torch.bfloat16).float().numpy())
    nan = orc.round_bf16(np.array([np.nan], np.float32))
    assert np.isnan(nan[0])
