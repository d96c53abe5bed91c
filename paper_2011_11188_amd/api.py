"""Tensor-level conveniences over the C ABI (argument marshalling only).

These derive sizes and leading dimensions from torch tensor shapes, allocate
outputs and workspaces with torch, and call the ``mdnn_*`` entry points.
"""
from __future__ import annotations

import ctypes as C
from typing import Optional, Sequence

from . import (ACT_NONE, BF16, F16, F32, LAYER_CONV, LAYER_FC, LAYER_MAXPOOL2, LOSS_MSE, LOSS_XENT,
               NN, NT, TN, ConvShape, LayerDesc, Scaler, TrainCfg, dtype_of, mdnn_conv2d_bwd_data,
               mdnn_conv2d_bwd_filter, mdnn_conv2d_bwd_filter_workspace, mdnn_conv2d_fwd,
               mdnn_gemm_mixed, mdnn_gemm_mixed_ws, mdnn_gemm_workspace, mdnn_gemm_split3,
               mdnn_gemm_split3_workspace, mdnn_net_activation, mdnn_net_output_grad, mdnn_net_bind, mdnn_net_create, mdnn_net_destroy, mdnn_net_sizes, mdnn_net_sync_lowp,
               mdnn_split_f16, mdnn_train_step, mdnn_train_step_async, mdnn_train_graph_create,
               mdnn_graph_launch, mdnn_graph_destroy, mdnn_conv2d_fwd_winograd,
               mdnn_conv2d_fwd_winograd_workspace, mdnn_conv2d_fwd_algo, mdnn_conv2d_fwd_algo_workspace)

__all__ = ["torch_dtype", "gemm", "split_f16", "gemm_split3", "conv_shape", "conv2d_fwd",
           "conv2d_fwd_winograd", "conv2d_fwd_algo", "conv2d_bwd_data", "conv2d_bwd_filter", "make_scaler", "read_scaler", "Net", "StepGraph"]


def torch_dtype(code: int):
    import torch
    return {F32: torch.float32, F16: torch.float16, BF16: torch.bfloat16}[code]


def gemm(layout: int, A, B, out_dtype=None, bias=None, act: int = ACT_NONE, mask=None,
         alpha: float = 1.0, beta: float = 0.0, Cm=None, out=None, stream=None, workspace=None,
         nonfinite=None):
    """D = epi(alpha op(A) op(B) + beta C) for row-major 2-D tensors A, B.
    workspace: None (mdnn_gemm_mixed), True (allocate what
    mdnn_gemm_workspace asks for) or a device byte tensor (mdnn_gemm_mixed_ws).
    nonfinite: a device int32 tensor set to 1 when a stored value of the fp32
    D is Inf or NaN (mdnn_gemm_mixed_ws; implies a workspace, empty if None)."""
    import torch
    if layout == TN:
        K, M = A.shape
    else:
        M, K = A.shape
    N = B.shape[0] if layout == NT else B.shape[1]
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype or torch.float32, device=A.device)
    args = (layout, M, N, K, alpha, A, A.stride(0), B, B.stride(0), dtype_of(A), beta, Cm,
            Cm.stride(0) if Cm is not None else 0, out, out.stride(0), dtype_of(out), bias,
            act, mask, mask.stride(0) if mask is not None else 0)
    if workspace is None and nonfinite is None:
        mdnn_gemm_mixed(*args, stream)
        return out
    if workspace is True:
        nb = mdnn_gemm_workspace(dtype_of(A), M, N, K)
        workspace = torch.empty((max(nb, 16),), dtype=torch.uint8, device=A.device)
    mdnn_gemm_mixed_ws(*args, workspace, workspace.numel() if workspace is not None else 0, stream,
                       nonfinite=nonfinite)
    return out


def split_f16(x, scale: float = 1.0, stream=None, scale_out=None):
    """(hi, lo) fp16 tensors of the two-term split of a 2-D fp32 tensor.
    scale 0 lets the library choose the power of two on the device; it is
    written to ``scale_out`` (a one-element fp32 device tensor, allocated when
    not given, returned as the third value)."""
    import torch
    rows, cols = x.shape
    hi = torch.empty((rows, cols), dtype=torch.float16, device=x.device)
    lo = torch.empty_like(hi)
    if scale == 0.0 and scale_out is None:
        scale_out = torch.empty((1,), dtype=torch.float32, device=x.device)
    mdnn_split_f16(rows, cols, x, x.stride(0), scale, scale_out, hi, cols, lo, cols, stream)
    return (hi, lo, scale_out) if scale == 0.0 else (hi, lo)


def gemm_split3(layout: int, A, B, a_scale: float = 1.0, b_scale: float = 1.0, alpha: float = 1.0,
                beta: float = 0.0, Cm=None, out=None, stream=None):
    """fp32 D = alpha op(A) op(B) + beta C through three fp16 MFMA products
    (a scale of 0: chosen on the device from the operand's largest magnitude)."""
    import torch
    if layout == TN:
        K, M = A.shape
    else:
        M, K = A.shape
    N = B.shape[0] if layout == NT else B.shape[1]
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=A.device)
    ws_bytes = mdnn_gemm_split3_workspace(M, N, K)
    ws = torch.empty((max(ws_bytes, 256),), dtype=torch.uint8, device=A.device)
    mdnn_gemm_split3(layout, M, N, K, alpha, A, A.stride(0), a_scale, B, B.stride(0), b_scale, beta, Cm,
                     Cm.stride(0) if Cm is not None else 0, out, out.stride(0), ws, ws_bytes, stream)
    return out


def conv_shape(x_shape: Sequence[int], c_out: int, r: int, s: int, pad: int) -> ConvShape:
    n, h, w, c = x_shape
    return ConvShape(n, h, w, c, c_out, r, s, pad)


def conv2d_fwd(x, w, pad: int, bias=None, act: int = ACT_NONE, out_dtype=None, stream=None):
    import torch
    k, r, s, c = w.shape
    sh = conv_shape(x.shape, k, r, s, pad)
    ho, wo = sh.h + 2 * pad - r + 1, sh.w + 2 * pad - s + 1
    y = torch.empty((sh.n, ho, wo, k), dtype=out_dtype or x.dtype, device=x.device)
    mdnn_conv2d_fwd(sh, x, w, dtype_of(x), bias, act, y, dtype_of(y), stream)
    return y


def conv2d_fwd_algo(x, w, pad: int, algo: int, bias=None, act: int = ACT_NONE, out_dtype=None, workspace=None,
                    stream=None):
    """conv2d_fwd through a chosen algorithm (CONV_AUTO: the library's
    per-layer choice for the given workspace; a workspace of the algorithm's
    size is allocated when none is given)."""
    import torch
    k, r, s, c = w.shape
    sh = conv_shape(x.shape, k, r, s, pad)
    ho, wo = sh.h + 2 * pad - r + 1, sh.w + 2 * pad - s + 1
    y = torch.empty((sh.n, ho, wo, k), dtype=out_dtype or x.dtype, device=x.device)
    io = dtype_of(x)
    if workspace is None:
        need = mdnn_conv2d_fwd_algo_workspace(sh, io, algo)
        workspace = torch.empty((max(need, 256),), dtype=torch.uint8, device=x.device)
    mdnn_conv2d_fwd_algo(sh, x, w, io, bias, act, y, dtype_of(y), algo, workspace, workspace.numel(), stream)
    return y


def conv2d_fwd_winograd(x, w, pad: int, bias=None, act: int = ACT_NONE, out_dtype=None, workspace=None,
                        stream=None):
    """conv2d_fwd through Winograd F(2x2, 3x3) (3x3 filters, fp16 / bf16)."""
    import torch
    k, r, s, c = w.shape
    sh = conv_shape(x.shape, k, r, s, pad)
    ho, wo = sh.h + 2 * pad - r + 1, sh.w + 2 * pad - s + 1
    y = torch.empty((sh.n, ho, wo, k), dtype=out_dtype or x.dtype, device=x.device)
    nb = mdnn_conv2d_fwd_winograd_workspace(sh, dtype_of(x))
    if workspace is None:
        workspace = torch.empty((max(nb, 256),), dtype=torch.uint8, device=x.device)
    mdnn_conv2d_fwd_winograd(sh, x, w, dtype_of(x), bias, act, y, dtype_of(y), workspace, workspace.numel(), stream)
    return y


def conv2d_bwd_data(dy, w, pad: int, h: int, wd: int, mask=None, out_dtype=None, stream=None):
    import torch
    k, r, s, c = w.shape
    sh = ConvShape(dy.shape[0], h, wd, c, k, r, s, pad)
    dx = torch.empty((sh.n, h, wd, c), dtype=out_dtype or dy.dtype, device=dy.device)
    mdnn_conv2d_bwd_data(sh, dy, w, dtype_of(dy), mask, dx, dtype_of(dx), stream)
    return dx


def conv2d_bwd_filter(x, dy, r: int, s: int, pad: int, with_db: bool = True, stream=None):
    import torch
    n, h, wd, c = x.shape
    k = dy.shape[3]
    sh = ConvShape(n, h, wd, c, k, r, s, pad)
    dw = torch.empty((k, r, s, c), dtype=torch.float32, device=x.device)
    db = torch.empty((k,), dtype=torch.float32, device=x.device) if with_db else None
    ws_bytes = mdnn_conv2d_bwd_filter_workspace(sh, dtype_of(x))
    ws = torch.empty((max(ws_bytes, 16),), dtype=torch.uint8, device=x.device)
    mdnn_conv2d_bwd_filter(sh, x, dy, dtype_of(x), dw, db, ws, ws_bytes, stream)
    return dw, db


def make_scaler(scale: float, growth_interval: int = 2000, growth: float = 2.0,
                backoff: float = 0.5, min_scale: float = 1.0, device="cuda"):
    """A device copy of an mdnn_scaler_t (32 bytes)."""
    import torch
    s = Scaler(scale, 0, 0, growth_interval, growth, backoff, min_scale, 0)
    raw = bytes(memoryview(s))
    return torch.frombuffer(bytearray(raw), dtype=torch.uint8).to(device)


def read_scaler(t) -> dict:
    raw = bytes(t.cpu().numpy().tobytes())
    s = Scaler.from_buffer_copy(raw)
    return {f: getattr(s, f) for f, _ in Scaler._fields_}


class Net:
    """A bound train-step handle: parameter, gradient, momentum, low-precision
    and workspace buffers are torch allocations owned by this object."""

    def __init__(self, layers, batch: int, dtype: int, loss: int, lr: float,
                 momentum: float = 0.0, loss_scaling: bool = False, init_scale: float = 1.0,
                 n_classes: int = 10, device="cuda", shared_master=None, fuse_update: bool = False):
        """shared_master: another Net's `master` tensor to bind instead of a
        private one (asynchronous workers; step with step_async only).
        fuse_update: the train config's fuse_update (eligible FC layers
        updated inside their weight-gradient products)."""
        import torch
        descs = [LayerDesc(l.kind, l.act, l.c_in, l.h, l.w, l.c_out, l.r, l.s, l.pad) for l in layers]
        self.cfg = TrainCfg(dtype, loss, lr, momentum, 1 if loss_scaling else 0,
                            n_classes if loss == LOSS_XENT else 0, 1 if fuse_update else 0)
        self.handle = mdnn_net_create(descs, batch, self.cfg)
        self.batch = batch
        self.dtype = dtype
        self.n_params, self.ws_bytes = mdnn_net_sizes(self.handle)
        dev = torch.device(device)
        if shared_master is not None:
            if shared_master.numel() != self.n_params or shared_master.dtype != torch.float32:
                raise ValueError("shared_master must be fp32 with this net's parameter count")
            self.master = shared_master
        else:
            self.master = torch.zeros(self.n_params, dtype=torch.float32, device=dev)
        self.grads = torch.zeros(self.n_params, dtype=torch.float32, device=dev)
        self.mom = torch.zeros(self.n_params, dtype=torch.float32, device=dev) if momentum else None
        self.lowp = (torch.zeros(self.n_params, dtype=torch_dtype(dtype), device=dev)
                     if dtype != F32 else None)
        self.ws = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=dev)
        self.scaler = make_scaler(init_scale, device=dev) if loss_scaling else None
        self.loss = torch.zeros(1, dtype=torch.float32, device=dev)
        mdnn_net_bind(self.handle, self.master, self.grads, self.mom, self.lowp, self.ws,
                      self.ws.numel(), self.scaler)

    def set_params(self, params, stream=None):
        """Copy fp32 master parameters (any array-like) and derive the
        low-precision working copy."""
        import torch
        self.master.copy_(torch.as_tensor(params, dtype=torch.float32))
        mdnn_net_sync_lowp(self.handle, stream)

    def step(self, x, target, loss_out=None, stream=None):
        out = self.loss if loss_out is None else loss_out
        mdnn_train_step(self.handle, x, target, out, stream)
        return out

    def record_step(self, x, target, loss_out=None) -> "StepGraph":
        """Record one step on these exact buffers into a HIP graph (see
        mdnn_train_graph_create); replay it with .launch()."""
        out = self.loss if loss_out is None else loss_out
        return StepGraph(mdnn_train_graph_create(self.handle, x, target, out), (self, x, target, out))

    def step_async(self, x, target, loss_out=None, stream=None):
        """Asynchronous step (section 3.1) on a master vector shared with other
        workers: see mdnn_train_step_async."""
        out = self.loss if loss_out is None else loss_out
        mdnn_train_step_async(self.handle, x, target, out, stream)
        return out

    def activation_ptr(self, i: int) -> Optional[int]:
        return mdnn_net_activation(self.handle, i)

    def output_grad_ptr(self, which: int) -> Optional[int]:
        return mdnn_net_output_grad(self.handle, which)

    def close(self):
        if getattr(self, "handle", None):
            mdnn_net_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class StepGraph:
    """A recorded train step.  Holds references to the net and the buffers
    the graph reads and writes, so they outlive it."""

    def __init__(self, handle: int, keep):
        self.handle = handle
        self._keep = keep

    def launch(self, stream=None):
        mdnn_graph_launch(self.handle, stream)

    def close(self):
        if getattr(self, "handle", None):
            mdnn_graph_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
