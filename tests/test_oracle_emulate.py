"""Pins of the oracle's emulate mode: the storage roundings of a
mixed-precision SGD step (section 3.2: 16-bit storage, fp32 accumulation and
fp32 master weights; section 3.1: the SGD update).

Two one-unit nets (FC 1->1 with ReLU, FC 1->1, MSE, batch 1, loss scale 8,
momentum 1/2, lr 1/16), one in fp16 and one in bfloat16, are stepped once and
every stored value is compared with a value derived by hand below.  The inputs
are chosen so that each storage rounding point changes a later value:

  x      not representable: the stored input x_lp differs from x, and the
         weight gradient of the first layer is formed from x_lp;
  a1     the hidden pre-activation is not representable: the stored
         activation a1 (and so the output and the loss) depends on it;
  dz     S * dL/dout is not representable: the second layer's gradients are
         formed from the rounded dz;
  dx     dz * w2 is not representable: the first layer's gradients are formed
         from the rounded dx;
  dW     x_lp * dx and a1 * dz are fp32 numbers that are not 16-bit numbers:
         the gradients stay in fp32;
  w_lp   the updated fp32 weights are not 16-bit numbers: the working copy is
         their rounding.

With u the storage spacing at 1 (fp16: 2^-10, bf16: 2^-7), both cases follow
the same derivation (S = 8, t = 0, B = 1, all products exact in fp64):
  x = 1 + 3u/4                       -> x_lp = 1 + u           (3/4 ulp rounds up)
  w1 = w2 = 1 + u, b1 = u/4, b2 = 0  (w_lp = w, biases from fp32 master)
  z1 = (1+u)^2 + u/4 = 1 + 2.25u + u^2 -> a1 = 1 + 2u         (0.25 ulp rounds down)
  out = a1 * w2 = 1 + 3u + 2u^2      (fp32-exact)
  L = out^2                           (unscaled mean over B = 1)
  S * 2 * out = 16 + 48u + 32u^2     -> dz = 16 + 48u         (spacing 16u at 16)
  g_w2 = a1 * dz = 16 + 80u + 96u^2  (fp32-exact, not a 16-bit number)
  g_b2 = dz = 16 + 48u
  dz * w2 = 16 + 64u + 48u^2         -> dx = 16 + 64u         (a1 > 0: not masked)
  g_w1 = x_lp * dx = 16 + 80u + 64u^2
  g_b1 = dx = 16 + 64u
  v = g / S (v0 = 0), w <- w - v / 16 (all fp32-exact)
  w1 = 7/8 + u - 5u/8 - u^2/2, w2 = 7/8 + u - 5u/8 - 3u^2/4
  -> w_lp(w1) = w_lp(w2) = 7/8 + u/2 (spacing u/2 below 1; 0.75 ulp rounds up)
A plausible slip at any one rounding point (a dropped rounding, or a
gradient rounded to 16 bits) changes at least one of these numbers.

The invariant tests check on random nets that every stored activation,
loss gradient and backward-data value is a 16-bit number, that the weight
gradients are fp32 numbers and mostly not 16-bit ones, and that the master
weights and momentum stay fp32 numbers.
"""
import numpy as np
import pytest

import workloads as W
from oracle import train
from oracle.rounding import round_to


def _one_unit_net(dtype: str):
    u = 2.0 ** -10 if dtype == "f16" else 2.0 ** -7
    layers = (W.Layer(W.FC, 1, c_out=1, act=W.ACT_RELU), W.Layer(W.FC, 1, c_out=1))
    params = np.array([1 + u, u / 4, 1 + u, 0.0])  # w1, b1, w2, b2
    net = train.OracleNet(layers, 1, dtype, W.LOSS_MSE, lr=2.0 ** -4, momentum=0.5,
                          loss_scaling=True, init_scale=8.0, params=params)
    return net, u


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_hand_derived_step(dtype):
    net, u = _one_unit_net(dtype)
    x = np.array([[1 + 0.75 * u]])
    t = np.array([[0.0]])

    acts, args, out = net.forward(x)
    assert acts[0][0, 0] == 1 + u                          # stored input
    assert acts[1][0, 0] == 1 + 2 * u                      # stored hidden activation
    assert out[0, 0] == 1 + 3 * u + 2 * u * u              # fp32 output
    loss, dz = net.loss_and_grad(out, t, 8.0)
    assert loss == (1 + 3 * u + 2 * u * u) ** 2
    assert dz[0, 0] == 16 + 48 * u                         # stored scaled loss gradient
    trace = []
    g = net.backward(acts, args, dz, trace=trace)
    assert trace[0][0, 0] == 16 + 64 * u                   # stored backward-data of layer 2
    want_g = [16 + 80 * u + 64 * u * u, 16 + 64 * u, 16 + 80 * u + 96 * u * u, 16 + 48 * u]
    assert g.tolist() == want_g                            # w1, b1, w2, b2 in fp32

    net2, _ = _one_unit_net(dtype)
    assert net2.step(x, t) == loss
    want_v = [v / 8 for v in want_g]
    want_w = [1 + u - want_v[0] / 16, u / 4 - want_v[1] / 16, 1 + u - want_v[2] / 16, -want_v[3] / 16]
    assert want_w[0] == 0.875 + u - 5 * u / 8 - u * u / 2
    assert want_w[2] == 0.875 + u - 5 * u / 8 - 3 * u * u / 4
    assert net2.v32.tolist() == want_v
    assert net2.w32.tolist() == want_w
    assert net2.w_lp()[[0, 2]].tolist() == [0.875 + u / 2, 0.875 + u / 2]
    assert net2.scaler["scale"] == 8.0 and net2.scaler["good_steps"] == 1


def _random_net(dtype: str, conv: bool, seed: int):
    g = np.random.default_rng(seed)
    if conv:
        layers = (W.Layer(W.CONV, 2, 6, 6, 4, 3, 3, 1, W.ACT_RELU),
                  W.Layer(W.MAXPOOL2, 4, 6, 6, 4),
                  W.Layer(W.CONV, 4, 3, 3, 4, 3, 3, 1, W.ACT_RELU),
                  W.Layer(W.FC, 36, c_out=5))
        in_f, loss = 72, W.LOSS_XENT
    else:
        layers = (W.Layer(W.FC, 24, c_out=32, act=W.ACT_RELU),
                  W.Layer(W.FC, 32, c_out=32, act=W.ACT_RELU),
                  W.Layer(W.FC, 32, c_out=1))
        in_f, loss = 24, W.LOSS_MSE
    n = sum(train.OracleNet._n_weight(l) + (l.c_out if l.kind != W.MAXPOOL2 else 0) for l in layers)
    p = round_to(g.standard_normal(n) * 0.4, "f32")
    net = train.OracleNet(layers, 6, dtype, loss, lr=0.1, momentum=0.9,
                          loss_scaling=True, init_scale=2.0 ** 6, params=p)
    x = g.standard_normal((6, in_f))
    t = g.integers(0, 5, 6) if conv else g.standard_normal((6, 1))
    return net, x, t


def _is(fmt, a):
    a = np.asarray(a, np.float64)
    return np.array_equal(round_to(a, fmt), a)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("conv", [False, True])
def test_storage_points_are_representable(dtype, conv):
    net, x, t = _random_net(dtype, conv, 11 + conv)
    assert not _is(dtype, x)                  # the raw input is not a 16-bit array ...
    acts, args, out = net.forward(x)
    assert _is(dtype, acts[0])                # ... the stored one is
    for a in acts[1:-1]:
        assert _is(dtype, a)                  # hidden activations (and pooled ones)
    assert _is("f32", out) and not _is(dtype, out)   # the output stays fp32
    loss, dz = net.loss_and_grad(out, t, net.scaler["scale"])
    assert _is(dtype, dz)
    trace = []
    g = net.backward(acts, args, dz, trace=trace)
    assert len(trace) == sum(1 for i, l in enumerate(net.layers) if i > 0 and l.kind != W.MAXPOOL2)
    for d in trace:
        assert _is(dtype, d)                  # every stored backward-data result
    assert _is("f32", g)
    # weight and bias gradients are not rounded to the storage type
    assert np.mean(round_to(g, dtype) != g) > 0.5
    db = np.concatenate([g[bo:bo + nb] for (_, bo, _, nb) in net.offsets if nb])
    assert np.mean(round_to(db, dtype) != db) > 0.5
    net.step(x, t)
    assert _is("f32", net.w32) and _is("f32", net.v32)
    assert not _is(dtype, net.w32)
