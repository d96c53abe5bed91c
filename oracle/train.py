"""fp64 oracle of one minibatch SGD step of a fixed layer chain.

Forward pass, loss, reverse-mode backpropagation (section 2.1) and the SGD
update (section 3.1), with the storage roundings of a mixed-precision step
(section 3.2: low-precision operands, fp32 accumulation, fp32 master weights).

Two modes:
* ``emulate``: round to the storage type at exactly the points where the step
  stores a tensor (list below); everything between two storage points is
  exact fp64.
* ``exact``: no rounding at all (used for finite-difference checks).

Storage points (``lp`` is the workload's storage type; fp32 workloads have
lp = fp32):
  x_lp = lp(x)                    the input batch
  w_lp = lp(w32)                  working weights, re-derived after each update
  a_l  = lp(act(acc + b32))       hidden activations (bias is fp32 master)
  out  = f32(acc + b32)           last layer output (logits / regression)
  dz   = lp(S * dL/dout)          loss gradient, scaled by the loss scale S
  dx   = lp((dz W^T) * [a_in>0])  backward-data, ReLU mask of the layer input
  dW, db = f32(...)               weight / bias gradients, straight from fp64
  w32, v32 = f32(update)          master weights and momentum
Max pooling only selects stored values (no rounding).

Test infrastructure only (see the package header).
"""
from __future__ import annotations

from typing import List, Optional

import numpy as np

from . import ops
from .rounding import round_to

FC, CONV, MAXPOOL2 = 0, 1, 2
ACT_RELU = 1
LOSS_XENT, LOSS_MSE = 0, 1


class OracleNet:
    """Mirrors a layer chain description with fields kind, c_in, h, w, c_out,
    r, s, pad, act (see ``workloads.Layer``)."""

    def __init__(self, layers, batch: int, dtype: str, loss: int, lr: float,
                 momentum: float = 0.0, loss_scaling: bool = False,
                 init_scale: float = 1.0, params: Optional[np.ndarray] = None,
                 mode: str = "emulate"):
        self.layers = list(layers)
        self.batch = batch
        self.lp = dtype
        self.loss_kind = loss
        self.lr = lr
        self.momentum = momentum
        self.mode = mode
        self.offsets = []
        off = 0
        for l in self.layers:
            nw = self._n_weight(l)
            nb = l.c_out if l.kind in (FC, CONV) else 0
            self.offsets.append((off, off + nw, nw, nb))
            off += nw + nb
        self.n_params = off
        self.w32 = np.zeros(off) if params is None else np.asarray(params, np.float64).copy()
        self.v32 = np.zeros(off) if momentum != 0.0 else None
        self.scaler = ops.new_scaler(init_scale) if loss_scaling else None
        # a layer's input is "post-ReLU" when it comes from a ReLU layer directly
        # or through max pooling of a ReLU output
        self.input_relu: List[bool] = []
        prev = False
        for l in self.layers:
            self.input_relu.append(prev)
            if l.kind == MAXPOOL2:
                pass  # pooling keeps the property of its input
            else:
                prev = l.act == ACT_RELU

    @staticmethod
    def _n_weight(l) -> int:
        if l.kind == FC:
            return l.c_in * l.c_out
        if l.kind == CONV:
            return l.c_out * l.r * l.s * l.c_in
        return 0

    # storage rounding helpers
    def R(self, x):
        return x if self.mode == "exact" else round_to(x, self.lp)

    def R32(self, x):
        return x if self.mode == "exact" else round_to(x, "f32")

    def w_lp(self) -> np.ndarray:
        return self.R(self.w32)

    def _wb(self, wl: np.ndarray, i: int, w32: Optional[np.ndarray] = None):
        l = self.layers[i]
        wo, bo, nw, nb = self.offsets[i]
        if l.kind == FC:
            w = wl[wo:wo + nw].reshape(l.c_in, l.c_out)
        else:
            w = wl[wo:wo + nw].reshape(l.c_out, l.r, l.s, l.c_in)
        return w, (self.w32 if w32 is None else w32)[bo:bo + nb]

    # -- forward / backward -------------------------------------------------
    def forward(self, x: np.ndarray, wl: Optional[np.ndarray] = None,
                w32: Optional[np.ndarray] = None):
        """Returns (stored activations a_0..a_L, pool argmaxes, output).  The
        biases come from the fp32 weights w32 (default: the current ones)."""
        wl = self.w_lp() if wl is None else wl
        b = self.batch
        a = self.R(np.asarray(x, np.float64).reshape(b, -1))
        acts, args = [a], {}
        n_l = len(self.layers)
        for i, l in enumerate(self.layers):
            last = i == n_l - 1
            if l.kind == FC:
                w, bias = self._wb(wl, i, w32)
                z = a.reshape(b, -1) @ w + bias
            elif l.kind == CONV:
                w, bias = self._wb(wl, i, w32)
                z = ops.conv2d_fwd(a.reshape(b, l.h, l.w, l.c_in), w, l.pad) + bias
            else:
                z, args[i] = ops.maxpool2_fwd(a.reshape(b, l.h, l.w, l.c_in))
            if l.kind != MAXPOOL2 and l.act == ACT_RELU:
                z = ops.relu(z)
            if l.kind == MAXPOOL2:
                a = z
            else:
                a = self.R32(z) if last else self.R(z)
            acts.append(a)
        return acts, args, acts[-1].reshape(b, -1)

    def loss_and_grad(self, out: np.ndarray, target: np.ndarray, scale: float):
        if self.loss_kind == LOSS_XENT:
            loss, dz = ops.softmax_xent(out, target, scale)
        else:
            loss, dz = ops.mse_loss(out, np.asarray(target, np.float64).reshape(out.shape), scale)
        return loss, self.R(dz)

    def backward(self, acts, args, dz: np.ndarray, wl: Optional[np.ndarray] = None,
                 trace: Optional[list] = None) -> np.ndarray:
        """Gradient of the loss (times the loss scale) w.r.t. the flat params.
        ``trace``, when given, receives each stored backward-data result (the
        gradient w.r.t. a layer's input, after the ReLU mask and the storage
        rounding), last layer first."""
        wl = self.w_lp() if wl is None else wl
        b = self.batch
        g = np.zeros(self.n_params)
        for i in range(len(self.layers) - 1, -1, -1):
            l = self.layers[i]
            a_in = acts[i]
            wo, bo, nw, nb = self.offsets[i]
            dx = None
            if l.kind == FC:
                w, _ = self._wb(wl, i)
                a2 = a_in.reshape(b, -1)
                dz2 = dz.reshape(b, -1)
                g[wo:wo + nw] = self.R32(a2.T @ dz2).ravel()
                g[bo:bo + nb] = self.R32(dz2.sum(axis=0))
                if i > 0:
                    dx = dz2 @ w.T
            elif l.kind == CONV:
                w, _ = self._wb(wl, i)
                x4 = a_in.reshape(b, l.h, l.w, l.c_in)
                dz4 = dz.reshape(b, l.h, l.w, l.c_out)
                g[wo:wo + nw] = self.R32(ops.conv2d_bwd_filter(x4, dz4, l.pad, l.r, l.s)).ravel()
                g[bo:bo + nb] = self.R32(dz4.sum(axis=(0, 1, 2)))
                if i > 0:
                    dx = ops.conv2d_bwd_data(dz4, w, l.pad, l.h, l.w)
            else:
                ho, wo_ = l.h // 2, l.w // 2
                dz = ops.maxpool2_bwd(dz.reshape(b, ho, wo_, l.c_in), args[i], l.h, l.w)
                continue
            if dx is not None:
                dx = dx.reshape(a_in.shape)
                if self.input_relu[i]:
                    dx = np.where(a_in > 0.0, dx, 0.0)
                dz = self.R(dx)
                if trace is not None:
                    trace.append(dz)
        return g

    def step(self, x: np.ndarray, target: np.ndarray) -> float:
        """One SGD step; returns the (unscaled) loss of the forward pass."""
        wl = self.w_lp()
        acts, args, out = self.forward(x, wl)
        s = 1.0 if self.scaler is None else self.scaler["scale"]
        loss, dz = self.loss_and_grad(out, target, s)
        g = self.backward(acts, args, dz, wl)
        w, v, sc, _ = ops.sgd_update(self.w32, g, self.v32, self.lr, self.momentum, self.scaler)
        self.w32 = self.R32(w)
        self.v32 = None if v is None else self.R32(v)
        self.scaler = sc
        return loss

    def loss_only(self, x: np.ndarray, target: np.ndarray) -> float:
        _, _, out = self.forward(x)
        loss, _ = self.loss_and_grad(out, target, 1.0)
        return loss


def from_config(cfg, params: Optional[np.ndarray] = None, mode: str = "emulate",
                batch: Optional[int] = None) -> OracleNet:
    """Build from a ``workloads.TrainConfig``-like object."""
    return OracleNet(cfg.layers, cfg.batch if batch is None else batch, cfg.dtype, cfg.loss,
                     cfg.lr, cfg.momentum, cfg.loss_scaling, cfg.init_scale, params, mode)
