"""Pins of the oracle's asynchronous-SGD model (section 3.1, bounded staleness).

* Staleness 0 is plain SGD: the model's trajectory equals OracleNet.step's,
  bit for bit.
* The delayed recursion's stability on f(w) = a w^2 / 2, where it is the
  linear recurrence w_{t+1} = w_t - c w_{t-tau} (c = lr a): stable for
  c < 2 without delay, for c < 1 with a delay of one, for c < (sqrt(5)-1)/2
  with a delay of two (roots of its characteristic polynomial) -- a wrong
  delay index moves these thresholds.
* Full-batch delayed gradient descent on a linear least-squares problem
  converges to numpy's lstsq solution.
* With two workers the second update's loss is the loss of its batch at the
  initial weights (both workers read before either updates).
"""
import numpy as np
import pytest

import workloads as W
from oracle import async_sgd
from oracle.train import from_config


@pytest.mark.parametrize("tau, c, stable", [(0, 1.5, True), (0, 2.1, False), (1, 0.9, True),
                                            (1, 1.1, False), (2, 0.55, True), (2, 0.7, False)])
def test_delayed_quadratic_stability(tau, c, stable):
    ws = async_sgd.delayed_sgd(lambda w, t: w, np.array([1.0]), c, 400, tau)
    tail = abs(ws[-1][0])
    if stable:
        assert tail < 1e-3
    else:
        assert tail > 1e3


def test_delayed_least_squares_converges_to_lstsq():
    g = np.random.default_rng(3)
    a = g.standard_normal((40, 6))
    y = g.standard_normal(40)
    sol = np.linalg.lstsq(a, y, rcond=None)[0]
    grad = lambda w, t: a.T @ (a @ w - y) / 40  # noqa: E731
    lr = 0.5 / np.linalg.norm(a, 2) ** 2 * 40 / 3
    for tau in (0, 1, 3):
        ws = async_sgd.delayed_sgd(grad, np.zeros(6), lr, 3000, tau)
        assert np.max(np.abs(ws[-1] - sol)) < 1e-8


def test_staleness_zero_is_plain_sgd():
    cfg = W.mlp784_fp32()
    p = W.init_params(cfg)
    batches = [W.batch_inputs(cfg, s, rows=16) for s in range(6)]
    a = from_config(cfg, p, batch=16)
    b = from_config(cfg, p, batch=16)
    la = async_sgd.async_train(a, batches, workers=1)
    lb = [b.step(x, t) for x, t in batches]
    assert la == lb
    assert np.array_equal(a.w32, b.w32)


def test_workers_use_stale_weights():
    """With two workers the second update's gradient is taken at w_0 (both
    workers read before either updates): it equals plain SGD's first gradient
    on batch 1 evaluated at w_0."""
    cfg = W.mlp784_fp32()
    p = W.init_params(cfg)
    batches = [W.batch_inputs(cfg, s, rows=16) for s in range(2)]
    a = from_config(cfg, p, batch=16)
    la = async_sgd.async_train(a, batches, workers=2)
    ref = from_config(cfg, p, batch=16)
    l1 = ref.loss_only(*batches[1])        # loss of batch 1 at w_0
    assert la[1] == l1
    ref2 = from_config(cfg, p, batch=16)
    ref2.step(*batches[0])
    assert la[1] != ref2.loss_only(*batches[1])
