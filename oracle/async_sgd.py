"""Asynchronous SGD in the bounded-staleness model (test infrastructure only).

Section 3.1 describes asynchronous SGD: workers compute gradients from the
parameter values they happen to read, while other workers keep updating the
shared parameters without locks (Hogwild!-style), so each applied gradient
may be stale.  The execution is non-deterministic; the oracle fixes the
standard deterministic model of it: W workers take turns, update t is
applied by worker t mod W, and its gradient is taken at the parameters as
they were `staleness` updates earlier (staleness = W - 1 when every worker
reads the parameters at the start of its step and the other W - 1 workers
each apply one update before it finishes):

    w_{t+1} = w_t - lr * grad(w_{t - staleness}; batch_t)     (w_{s<0} = w_0)

With momentum each worker keeps its own velocity (v_k <- mu v_k + g), and
with loss scaling its own scaler, as the GPU workers do.

The GPU's real interleaving varies from run to run, so parity against this
model is statistical (loss after many updates); with one worker (staleness 0)
the model is plain SGD and parity is exact up to rounding.
"""
from __future__ import annotations

from typing import Callable, List, Sequence, Tuple

import numpy as np

from . import ops
from .train import OracleNet


def delayed_sgd(grad_fn: Callable[[np.ndarray, int], np.ndarray], w0: np.ndarray, lr: float,
                n_updates: int, staleness: int) -> List[np.ndarray]:
    """The recursion above for a gradient oracle grad_fn(w, t); returns the
    iterates w_0 .. w_n (exact arithmetic, no storage rounding)."""
    ws = [np.array(w0, dtype=np.float64)]
    for t in range(n_updates):
        w_read = ws[max(0, t - staleness)]
        ws.append(ws[-1] - lr * grad_fn(w_read, t))
    return ws


def async_train(net: OracleNet, batches: Sequence[Tuple[np.ndarray, np.ndarray]], workers: int,
                ) -> List[float]:
    """Train `net` (its master weights are the shared parameters) on
    `batches` in the model above with staleness workers - 1; worker
    t mod W takes update t.  Storage roundings as in OracleNet.step (the
    gradient step reads the working copy lp(w32) of the stale weights).
    Returns the loss of each update's forward pass."""
    staleness = workers - 1
    hist = [net.w32.copy()]
    vel = [None if net.v32 is None else np.zeros_like(net.w32) for _ in range(workers)]
    scalers = [None if net.scaler is None else dict(net.scaler) for _ in range(workers)]
    losses = []
    for t, (x, target) in enumerate(batches):
        k = t % workers
        w_read = hist[max(0, t - staleness)]
        wl = net.R(w_read)
        acts, args, out = net.forward(x, wl, w32=w_read)
        s = 1.0 if scalers[k] is None else scalers[k]["scale"]
        loss, dz = net.loss_and_grad(out, target, s)
        g = net.backward(acts, args, dz, wl)
        w, v, sc, _ = ops.sgd_update(net.w32, g, vel[k], net.lr, net.momentum, scalers[k])
        net.w32 = net.R32(w)
        vel[k] = None if v is None else net.R32(v)
        scalers[k] = sc
        hist.append(net.w32.copy())
        losses.append(loss)
    return losses
