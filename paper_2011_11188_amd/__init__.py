"""Python binding of libmdnn (MI355X / gfx950): argument marshalling only.

Every function named ``mdnn_*`` here calls the C entry point of the same name
in ``libmdnn.so`` (declared in ``include/mdnn.h``).  Pointer arguments accept
a torch tensor (its ``data_ptr()``), a raw integer address or ``None`` (NULL);
``stream=None`` means torch's current stream on the current device.  A
non-success status raises :class:`MdnnError`.  No computation happens in
Python and there is no fallback: importing this package raises when the HIP
library has not been built.

PyTorch is used only to allocate device memory and to name streams.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmdnn.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it with `python paper_2011_11188_amd/build.py` "
        "(the HIP path has no fallback)")

_lib = C.CDLL(LIB_PATH)

# enums (include/mdnn.h)
SUCCESS, ERR_NULL, ERR_SHAPE, ERR_LAYOUT, ERR_DTYPE, ERR_MISALIGNED, ERR_WORKSPACE, ERR_LAUNCH, \
    ERR_STATE = range(9)
F32, F16, BF16 = 0, 1, 2
NN, NT, TN = 0, 1, 2
ACT_NONE, ACT_RELU = 0, 1
LAYER_FC, LAYER_CONV, LAYER_MAXPOOL2 = 0, 1, 2
LOSS_XENT, LOSS_MSE = 0, 1
CONV_AUTO, CONV_IMPLICIT_GEMM, CONV_IM2COL_GEMM, CONV_WINOGRAD = 0, 1, 2, 3

_STATUS_NAMES = {0: "SUCCESS", 1: "ERR_NULL", 2: "ERR_SHAPE", 3: "ERR_LAYOUT", 4: "ERR_DTYPE",
                 5: "ERR_MISALIGNED", 6: "ERR_WORKSPACE", 7: "ERR_LAUNCH", 8: "ERR_STATE"}


class MdnnError(RuntimeError):
    def __init__(self, status: int, func: str, msg: str):
        super().__init__(f"{func}: {_STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class ConvShape(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("n", "h", "w", "c_in", "c_out", "r", "s", "pad")]


class Scaler(C.Structure):
    _fields_ = [("scale", C.c_float), ("good_steps", C.c_int32), ("overflow", C.c_int32),
                ("growth_interval", C.c_int32), ("growth", C.c_float), ("backoff", C.c_float),
                ("min_scale", C.c_float), ("reserved", C.c_int32)]


class LayerDesc(C.Structure):
    _fields_ = [("kind", C.c_int32), ("act", C.c_int32)] + \
        [(n, C.c_int64) for n in ("c_in", "h", "w", "c_out", "r", "s", "pad")]


class TrainCfg(C.Structure):
    _fields_ = [("dtype", C.c_int32), ("loss", C.c_int32), ("lr", C.c_float),
                ("momentum", C.c_float), ("loss_scaling", C.c_int32), ("n_classes", C.c_int32),
                ("fuse_update", C.c_int32)]


_vp, _i64, _f, _i = C.c_void_p, C.c_int64, C.c_float, C.c_int

_SIGS = {
    "mdnn_gemm_mixed": [_i, _i64, _i64, _i64, _f, _vp, _i64, _vp, _i64, _i, _f, _vp, _i64, _vp,
                        _i64, _i, _vp, _i, _vp, _i64, _vp],
    "mdnn_gemm_mixed_ws": [_i, _i64, _i64, _i64, _f, _vp, _i64, _vp, _i64, _i, _f, _vp, _i64, _vp,
                           _i64, _i, _vp, _i, _vp, _i64, _vp, C.c_size_t, _vp, _vp],
    "mdnn_gemm_tn_update": [_i64, _i64, _i64, _vp, _i64, _vp, _i64, _i, _vp, _vp, _vp, _i64, _f, _f, _vp, _vp],
    "mdnn_conv2d_fwd": [_vp, _vp, _vp, _i, _vp, _i, _vp, _i, _vp],
    "mdnn_conv2d_bwd_data": [_vp, _vp, _vp, _i, _vp, _vp, _i, _vp],
    "mdnn_conv2d_bwd_filter": [_vp, _vp, _vp, _i, _vp, _vp, _vp, C.c_size_t, _vp],
    "mdnn_conv2d_bwd_filter_noalloc": [_vp, _vp, _vp, _i, _vp, _vp, _vp],
    "mdnn_conv2d_fwd_winograd": [_vp, _vp, _vp, _i, _vp, _i, _vp, _i, _vp, C.c_size_t, _vp],
    "mdnn_conv2d_fwd_algo": [_vp, _vp, _vp, _i, _vp, _i, _vp, _i, _i, _vp, C.c_size_t, _vp],
    "mdnn_bias_act_fwd": [_i64, _i64, _vp, _vp, _i, _vp, _i, _vp],
    "mdnn_bias_act_bwd": [_i64, _i64, _vp, _vp, _i, _vp, _vp, _i, _vp, C.c_size_t, _vp],
    "mdnn_maxpool2_fwd": [_i64, _i64, _i64, _i64, _vp, _vp, _vp, _i, _vp],
    "mdnn_maxpool2_bwd": [_i64, _i64, _i64, _i64, _vp, _vp, _vp, _i, _vp],
    "mdnn_softmax_xent": [_i64, _i64, _vp, _i64, _vp, _vp, _vp, _vp, _i64, _i, _vp],
    "mdnn_mse_loss": [_i64, _i64, _vp, _vp, _vp, _vp, _vp, _i, _vp],
    "mdnn_sgd_update": [_i64, _vp, _vp, _vp, _vp, _i, _f, _f, _vp, _vp],
    "mdnn_cast": [_i64, _vp, _i, _vp, _i, _vp],
    "mdnn_sgd_update_async": [_i64, _vp, _vp, _vp, _f, _f, _vp, _vp],
    "mdnn_train_step_async": [_vp, _vp, _vp, _vp, _vp],
    "mdnn_split_f16": [_i64, _i64, _vp, _i64, _f, _vp, _vp, _i64, _vp, _i64, _vp],
    "mdnn_gemm_split3": [_i, _i64, _i64, _i64, _f, _vp, _i64, _f, _vp, _i64, _f, _f, _vp, _i64, _vp,
                         _i64, _vp, C.c_size_t, _vp],
    "mdnn_net_create": [_vp, C.c_int32, _i64, _vp, _vp],
    "mdnn_net_sizes": [_vp, _vp, _vp],
    "mdnn_net_bind": [_vp, _vp, _vp, _vp, _vp, _vp, C.c_size_t, _vp],
    "mdnn_net_sync_lowp": [_vp, _vp],
    "mdnn_train_step": [_vp, _vp, _vp, _vp, _vp],
    "mdnn_train_graph_create": [_vp, _vp, _vp, _vp, _vp],
    "mdnn_graph_launch": [_vp, _vp],
}
for _name, _args in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = C.c_int
_lib.mdnn_conv2d_bwd_filter_workspace.argtypes = [_vp, _i]
_lib.mdnn_conv2d_bwd_filter_workspace.restype = C.c_size_t
_lib.mdnn_conv2d_bwd_filter_noalloc_max_workspace.argtypes = []
_lib.mdnn_conv2d_bwd_filter_noalloc_max_workspace.restype = C.c_size_t
_lib.mdnn_conv2d_fwd_winograd_workspace.argtypes = [_vp, _i]
_lib.mdnn_conv2d_fwd_winograd_workspace.restype = C.c_size_t
_lib.mdnn_conv2d_fwd_algo_workspace.argtypes = [_vp, _i, _i]
_lib.mdnn_conv2d_fwd_algo_workspace.restype = C.c_size_t
_lib.mdnn_conv2d_fwd_choose.argtypes = [_vp, _i, C.c_size_t]
_lib.mdnn_conv2d_fwd_choose.restype = _i
_lib.mdnn_gemm_workspace.argtypes = [_i, _i64, _i64, _i64]
_lib.mdnn_gemm_workspace.restype = C.c_size_t
_lib.mdnn_gemm_split3_workspace.argtypes = [_i64, _i64, _i64]
_lib.mdnn_gemm_split3_workspace.restype = C.c_size_t
_lib.mdnn_bias_act_bwd_workspace.argtypes = [_i64, _i64]
_lib.mdnn_bias_act_bwd_workspace.restype = C.c_size_t
_lib.mdnn_last_error.restype = C.c_char_p
_lib.mdnn_version.restype = C.c_char_p
_lib.mdnn_net_activation.argtypes = [_vp, C.c_int32]
_lib.mdnn_net_activation.restype = _vp
_lib.mdnn_net_output_grad.argtypes = [_vp, C.c_int32]
_lib.mdnn_net_output_grad.restype = _vp
_lib.mdnn_net_destroy.argtypes = [_vp]
_lib.mdnn_net_destroy.restype = None
_lib.mdnn_graph_destroy.argtypes = [_vp]
_lib.mdnn_graph_destroy.restype = None
_lib.mdnn_set_gemm_tile.argtypes = [_i]
_lib.mdnn_set_gemm_tile.restype = _i


def _p(x) -> Optional[int]:
    """Pointer of a tensor / ctypes object / int, or None for NULL."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if isinstance(x, C.Structure):
        return C.addressof(x)
    return C.cast(x, C.c_void_p).value


def _s(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _call(name: str, *args) -> int:
    st = getattr(_lib, name)(*args)
    if st != SUCCESS:
        raise MdnnError(st, name, _lib.mdnn_last_error().decode())
    return st


def dtype_of(t) -> int:
    import torch
    return {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16}[t.dtype]


def version() -> str:
    return _lib.mdnn_version().decode()


def last_error() -> str:
    return _lib.mdnn_last_error().decode()


def exported_symbols():
    return sorted(list(_SIGS) + ["mdnn_conv2d_bwd_filter_workspace", "mdnn_bias_act_bwd_workspace",
                                 "mdnn_conv2d_bwd_filter_noalloc_max_workspace",
                                 "mdnn_gemm_split3_workspace", "mdnn_gemm_workspace",
                                 "mdnn_conv2d_fwd_winograd_workspace", "mdnn_conv2d_fwd_algo_workspace",
                                 "mdnn_conv2d_fwd_choose",
                                 "mdnn_last_error",
                                 "mdnn_version", "mdnn_net_activation", "mdnn_net_output_grad", "mdnn_net_destroy",
                                 "mdnn_graph_destroy", "mdnn_set_gemm_tile"])


# ---------------------------------------------------------------------------
# one wrapper per entry point, same names and argument order as the C ABI
# ---------------------------------------------------------------------------

def mdnn_gemm_mixed(layout, M, N, K, alpha, A, lda, B, ldb, ab_type, beta, Cm, ldc, D, ldd,
                    d_type, bias=None, act=ACT_NONE, mask_src=None, ldm=0, stream=None):
    return _call("mdnn_gemm_mixed", layout, M, N, K, alpha, _p(A), lda, _p(B), ldb, ab_type, beta,
                 _p(Cm), ldc, _p(D), ldd, d_type, _p(bias), act, _p(mask_src), ldm, _s(stream))


def mdnn_set_gemm_tile(code: int) -> int:
    return _lib.mdnn_set_gemm_tile(code)


def mdnn_conv2d_fwd(shape: ConvShape, x, w, io_type, bias, act, y, y_type, stream=None):
    return _call("mdnn_conv2d_fwd", _p(shape), _p(x), _p(w), io_type, _p(bias), act, _p(y), y_type,
                 _s(stream))


def mdnn_conv2d_bwd_data(shape: ConvShape, dy, w, io_type, mask_src, dx, dx_type, stream=None):
    return _call("mdnn_conv2d_bwd_data", _p(shape), _p(dy), _p(w), io_type, _p(mask_src), _p(dx),
                 dx_type, _s(stream))


def mdnn_gemm_mixed_ws(layout, M, N, K, alpha, A, lda, B, ldb, ab_type, beta, Cm, ldc, D, ldd,
                       d_type, bias=None, act=ACT_NONE, mask_src=None, ldm=0, workspace=None, ws_bytes=0,
                       stream=None, nonfinite=None):
    return _call("mdnn_gemm_mixed_ws", layout, M, N, K, alpha, _p(A), lda, _p(B), ldb, ab_type, beta,
                 _p(Cm), ldc, _p(D), ldd, d_type, _p(bias), act, _p(mask_src), ldm, _p(workspace), ws_bytes,
                 _p(nonfinite), _s(stream))


def mdnn_gemm_tn_update(M, N, K, A, lda, B, ldb, ab_type, w32, v32, w_lp, ldw, lr, momentum, scaler=None,
                        stream=None):
    return _call("mdnn_gemm_tn_update", M, N, K, _p(A), lda, _p(B), ldb, ab_type, _p(w32), _p(v32), _p(w_lp),
                 ldw, lr, momentum, _p(scaler), _s(stream))


def mdnn_gemm_workspace(ab_type, M, N, K) -> int:
    return _lib.mdnn_gemm_workspace(ab_type, M, N, K)


def mdnn_conv2d_fwd_winograd(shape: ConvShape, x, w, io_type, bias, act, y, y_type, workspace, ws_bytes,
                             stream=None):
    return _call("mdnn_conv2d_fwd_winograd", _p(shape), _p(x), _p(w), io_type, _p(bias), act, _p(y), y_type,
                 _p(workspace), ws_bytes, _s(stream))


def mdnn_conv2d_fwd_algo(shape: ConvShape, x, w, io_type, bias, act, y, y_type, algo, workspace, ws_bytes,
                         stream=None):
    return _call("mdnn_conv2d_fwd_algo", _p(shape), _p(x), _p(w), io_type, _p(bias), act, _p(y), y_type, algo,
                 _p(workspace), ws_bytes, _s(stream))


def mdnn_conv2d_fwd_algo_workspace(shape: ConvShape, io_type, algo) -> int:
    return _lib.mdnn_conv2d_fwd_algo_workspace(_p(shape), io_type, algo)


def mdnn_conv2d_fwd_choose(shape: ConvShape, io_type, ws_bytes) -> int:
    return _lib.mdnn_conv2d_fwd_choose(_p(shape), io_type, ws_bytes)


def mdnn_conv2d_fwd_winograd_workspace(shape: ConvShape, io_type) -> int:
    return _lib.mdnn_conv2d_fwd_winograd_workspace(_p(shape), io_type)


def mdnn_conv2d_bwd_filter_workspace(shape: ConvShape, io_type) -> int:
    return _lib.mdnn_conv2d_bwd_filter_workspace(_p(shape), io_type)


def mdnn_conv2d_bwd_filter(shape: ConvShape, x, dy, io_type, dw, db, workspace, ws_bytes,
                           stream=None):
    return _call("mdnn_conv2d_bwd_filter", _p(shape), _p(x), _p(dy), io_type, _p(dw), _p(db),
                 _p(workspace), ws_bytes, _s(stream))


def mdnn_conv2d_bwd_filter_noalloc_max_workspace() -> int:
    return _lib.mdnn_conv2d_bwd_filter_noalloc_max_workspace()


def mdnn_conv2d_bwd_filter_noalloc(shape: ConvShape, x, dy, io_type, dw, db, stream=None):
    return _call("mdnn_conv2d_bwd_filter_noalloc", _p(shape), _p(x), _p(dy), io_type, _p(dw), _p(db),
                 _s(stream))


def mdnn_bias_act_fwd(rows, cols, x, bias, act, y, y_type, stream=None):
    return _call("mdnn_bias_act_fwd", rows, cols, _p(x), _p(bias), act, _p(y), y_type, _s(stream))


def mdnn_bias_act_bwd_workspace(rows, cols) -> int:
    return _lib.mdnn_bias_act_bwd_workspace(rows, cols)


def mdnn_bias_act_bwd(rows, cols, dy, y, act, dz, db, dtype, workspace=None, ws_bytes=0,
                      stream=None):
    return _call("mdnn_bias_act_bwd", rows, cols, _p(dy), _p(y), act, _p(dz), _p(db), dtype,
                 _p(workspace), ws_bytes, _s(stream))


def mdnn_maxpool2_fwd(n, h, w, c, x, y, argmax, dtype, stream=None):
    return _call("mdnn_maxpool2_fwd", n, h, w, c, _p(x), _p(y), _p(argmax), dtype, _s(stream))


def mdnn_maxpool2_bwd(n, h, w, c, dy, argmax, dx, dtype, stream=None):
    return _call("mdnn_maxpool2_bwd", n, h, w, c, _p(dy), _p(argmax), _p(dx), dtype, _s(stream))


def mdnn_softmax_xent(B, Cn, logits, ldl, labels, loss_scale, loss_out, dlogits, ldd, dlogits_type,
                      stream=None):
    return _call("mdnn_softmax_xent", B, Cn, _p(logits), ldl, _p(labels), _p(loss_scale),
                 _p(loss_out), _p(dlogits), ldd, dlogits_type, _s(stream))


def mdnn_mse_loss(B, O, y, t, loss_scale, loss_out, dy, dy_type, stream=None):
    return _call("mdnn_mse_loss", B, O, _p(y), _p(t), _p(loss_scale), _p(loss_out), _p(dy), dy_type,
                 _s(stream))


def mdnn_sgd_update(n, w32, g32, v32, w_lp, lp_type, lr, momentum, scaler, stream=None):
    return _call("mdnn_sgd_update", n, _p(w32), _p(g32), _p(v32), _p(w_lp), lp_type, lr, momentum,
                 _p(scaler), _s(stream))


def mdnn_cast(n, src, src_type, dst, dst_type, stream=None):
    return _call("mdnn_cast", n, _p(src), src_type, _p(dst), dst_type, _s(stream))


def mdnn_sgd_update_async(n, w32, g32, v32, lr, momentum, scaler=None, stream=None):
    return _call("mdnn_sgd_update_async", n, _p(w32), _p(g32), _p(v32), lr, momentum, _p(scaler),
                 _s(stream))


def mdnn_train_step_async(net, x, target, loss_out, stream=None):
    return _call("mdnn_train_step_async", net, _p(x), _p(target), _p(loss_out), _s(stream))


def mdnn_split_f16(rows, cols, x, ldx, scale, scale_out, hi, ldh, lo, ldl, stream=None):
    return _call("mdnn_split_f16", rows, cols, _p(x), ldx, scale, _p(scale_out), _p(hi), ldh, _p(lo), ldl,
                 _s(stream))


def mdnn_gemm_split3_workspace(M, N, K) -> int:
    return _lib.mdnn_gemm_split3_workspace(M, N, K)


def mdnn_gemm_split3(layout, M, N, K, alpha, A, lda, a_scale, B, ldb, b_scale, beta, Cm, ldc, D, ldd,
                     workspace, ws_bytes, stream=None):
    return _call("mdnn_gemm_split3", layout, M, N, K, alpha, _p(A), lda, a_scale, _p(B), ldb, b_scale,
                 beta, _p(Cm), ldc, _p(D), ldd, _p(workspace), ws_bytes, _s(stream))


def mdnn_net_create(layers, batch: int, cfg: TrainCfg) -> int:
    arr = (LayerDesc * len(layers))(*layers)
    h = C.c_void_p()
    _call("mdnn_net_create", C.addressof(arr), len(layers), batch, C.addressof(cfg), C.byref(h))
    return h.value


def mdnn_net_sizes(net: int):
    n = C.c_int64()
    ws = C.c_size_t()
    _call("mdnn_net_sizes", net, C.byref(n), C.byref(ws))
    return n.value, ws.value


def mdnn_net_bind(net, master_w, grads, momentum, lowp_w, workspace, ws_bytes, scaler):
    return _call("mdnn_net_bind", net, _p(master_w), _p(grads), _p(momentum), _p(lowp_w),
                 _p(workspace), ws_bytes, _p(scaler))


def mdnn_net_sync_lowp(net, stream=None):
    return _call("mdnn_net_sync_lowp", net, _s(stream))


def mdnn_train_step(net, x, target, loss_out, stream=None):
    return _call("mdnn_train_step", net, _p(x), _p(target), _p(loss_out), _s(stream))


def mdnn_net_activation(net, i: int) -> Optional[int]:
    return _lib.mdnn_net_activation(net, i)


def mdnn_net_output_grad(net, which: int) -> Optional[int]:
    return _lib.mdnn_net_output_grad(net, which)


def mdnn_net_destroy(net) -> None:
    _lib.mdnn_net_destroy(net)


def mdnn_train_graph_create(net, x, target, loss_out) -> int:
    """Returns the graph handle (an int)."""
    out = C.c_void_p()
    _call("mdnn_train_graph_create", net, _p(x), _p(target), _p(loss_out), C.byref(out))
    return out.value


def mdnn_graph_launch(graph, stream=None):
    return _call("mdnn_graph_launch", graph, _s(stream))


def mdnn_graph_destroy(graph) -> None:
    _lib.mdnn_graph_destroy(graph)


from .api import *  # noqa: E402,F401,F403  (tensor-level conveniences)
