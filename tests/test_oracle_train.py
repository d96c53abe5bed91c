"""Pins of the oracle's whole SGD step (forward, backprop, update).

* central finite differences of the loss in exact (unrounded) mode pin the
  backward chain, ReLU masks through max pooling included;
* uniform logits give loss = ln 10 for ten classes;
* power-of-two loss scales give bitwise-identical trajectories when nothing
  overflows or underflows;
* a forced overflow skips the update and halves the scale.
Whole-step numbers themselves have no worked example in the paper.
"""
import math

import numpy as np
import pytest

import workloads as W
from oracle import train
from oracle.rounding import round_to


def _fd_check(net, x, t, n_coords=60, eps=1e-4, seed=0):
    acts, args, out = net.forward(x)
    loss, dz = net.loss_and_grad(out, t, 1.0)
    g = net.backward(acts, args, dz)
    rs = np.random.default_rng(seed)
    idx = rs.choice(net.n_params, size=min(n_coords, net.n_params), replace=False)
    w0 = net.w32.copy()
    worst = 0.0
    for i in idx:
        net.w32 = w0.copy()
        net.w32[i] += eps
        lp = net.loss_only(x, t)
        net.w32 = w0.copy()
        net.w32[i] -= eps
        lm = net.loss_only(x, t)
        fd = (lp - lm) / (2 * eps)
        worst = max(worst, abs(fd - g[i]) / max(1e-3, abs(g[i]), abs(fd)))
    net.w32 = w0
    return worst


def test_fd_mlp_xent():
    layers = (W.Layer(W.FC, 8, c_out=5, act=W.ACT_RELU), W.Layer(W.FC, 5, c_out=3))
    g = np.random.default_rng(1)
    net = train.OracleNet(layers, 4, "f32", W.LOSS_XENT, 0.1, mode="exact")
    net.w32 = g.standard_normal(net.n_params) * 0.7
    x = g.standard_normal((4, 8))
    t = np.array([0, 2, 1, 2])
    assert _fd_check(net, x, t) < 1e-6


def test_fd_mlp_mse_deep():
    layers = (W.Layer(W.FC, 6, c_out=7, act=W.ACT_RELU), W.Layer(W.FC, 7, c_out=7, act=W.ACT_RELU),
              W.Layer(W.FC, 7, c_out=1))
    g = np.random.default_rng(2)
    net = train.OracleNet(layers, 5, "f32", W.LOSS_MSE, 0.1, mode="exact")
    net.w32 = g.standard_normal(net.n_params) * 0.6
    x = g.standard_normal((5, 6))
    t = g.standard_normal((5, 1))
    assert _fd_check(net, x, t) < 1e-6


def test_fd_conv_pool_net():
    layers = (W.Layer(W.CONV, 1, 6, 6, 2, 3, 3, 1, W.ACT_RELU),
              W.Layer(W.MAXPOOL2, 2, 6, 6, 2),
              W.Layer(W.CONV, 2, 3, 3, 3, 3, 3, 1, W.ACT_RELU),
              W.Layer(W.FC, 27, c_out=4))
    g = np.random.default_rng(3)
    net = train.OracleNet(layers, 3, "f32", W.LOSS_XENT, 0.1, mode="exact")
    net.w32 = g.standard_normal(net.n_params) * 0.8
    x = g.standard_normal((3, 36))
    t = np.array([1, 3, 0])
    assert _fd_check(net, x, t, n_coords=net.n_params) < 1e-6


def test_zero_last_layer_gives_ln10():
    cfg = W.mlp784_fp32()
    p = W.init_params(cfg)
    wo, bo = cfg.param_offsets()[1]
    p[wo:] = 0.0
    net = train.from_config(cfg, p)
    x, t = W.batch_inputs(cfg, 0)
    assert net.loss_only(x, t) == pytest.approx(math.log(10.0), abs=1e-15)


def _bf16_scaled_net(scale):
    layers = (W.Layer(W.FC, 16, c_out=12, act=W.ACT_RELU), W.Layer(W.FC, 12, c_out=10))
    g = np.random.default_rng(4)
    p = round_to(g.standard_normal(16 * 12 + 12 + 12 * 10 + 10) * 0.3, "f32")
    return train.OracleNet(layers, 8, "bf16", W.LOSS_XENT, 0.05, momentum=0.9,
                           loss_scaling=True, init_scale=scale, params=p)


def test_power_of_two_loss_scale_invariance():
    """bf16 has fp32's exponent range, so scaling by 2^16 commutes with every
    storage rounding: both trajectories are bitwise equal."""
    a, b = _bf16_scaled_net(1.0), _bf16_scaled_net(2.0 ** 16)
    g = np.random.default_rng(5)
    for step in range(5):
        x = g.random((8, 16))
        t = g.integers(0, 10, 8)
        la, lb = a.step(x, t), b.step(x, t)
        assert la == lb
        assert np.array_equal(a.w32, b.w32) and np.array_equal(a.v32, b.v32)


def test_forced_overflow_skips_step_and_halves_scale():
    layers = (W.Layer(W.FC, 32, c_out=16, act=W.ACT_RELU), W.Layer(W.FC, 16, c_out=1))
    g = np.random.default_rng(6)
    n = 32 * 16 + 16 + 16 + 1
    p = round_to(g.standard_normal(n) * 0.2, "f32")
    net = train.OracleNet(layers, 16, "f16", W.LOSS_MSE, 1e-3, momentum=0.9,
                          loss_scaling=True, init_scale=2.0 ** 40, params=p)
    x = g.standard_normal((16, 32))
    t = g.standard_normal((16, 1)) * 100.0
    w0 = net.w32.copy()
    net.step(x, t)                          # S * dL/dy overflows fp16 -> inf -> skip
    assert np.array_equal(net.w32, w0) and np.all(net.v32 == 0.0)
    assert net.scaler["scale"] == 2.0 ** 39 and net.scaler["good_steps"] == 0


def test_emulated_step_tracks_exact_step():
    """Storage rounding perturbs the loss only at the level of the storage
    precision (sanity of the rounding points, not a parity claim)."""
    cfg = W.lenet_bf16()
    small = train.from_config(cfg, W.init_params(cfg), batch=8)
    exact = train.from_config(cfg, W.init_params(cfg), mode="exact", batch=8)
    x, t = W.batch_inputs(cfg, 0, rows=8)
    le, lx = small.step(x, t), exact.step(x, t)
    assert abs(le - lx) / lx < 2e-2
    assert math.isfinite(le)
