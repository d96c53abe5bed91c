"""Forward convolution through the selectable algorithms (section 2.1: the
algorithm behind the operation is interchangeable per layer): the im2col +
GEMM comparator against the oracle (same bar as the implicit GEMM), the
automatic choice, and the dispatch to the implicit GEMM / Winograd entry
points (bitwise the same results as calling them directly)."""
import numpy as np
import pytest

import workloads as W
from oracle import ops
from oracle.rounding import decode
from tests.helpers import accum_bound, dev, host64, lowp_close, norm_max_err

pytestmark = pytest.mark.gpu
TOL = 1e-4


@pytest.mark.parametrize("dt", ["f16", "bf16", "f32"])
@pytest.mark.parametrize("shape", [(3, 9, 7, 16, 24, 3, 3, 1), (2, 6, 5, 3, 20, 5, 5, 2), (4, 8, 8, 64, 64, 3, 3, 1),
                                   (1, 5, 6, 8, 9, 3, 2, 0)])
def test_im2col_gemm_against_oracle(mdnn, dt, shape):
    import torch
    n, h, w, ci, co, r, s, pad = shape
    x = W.normal((n, h, w, ci), 71, 1, dt, 0.5)
    wt = W.normal((co, r, s, ci), 71, 2, dt, 0.3)
    b = W.normal((co,), 71, 3, "f32", 0.2)
    X, Wt = dev(x, dt), dev(wt, dt)
    y32 = mdnn.conv2d_fwd_algo(X, Wt, pad, mdnn.CONV_IM2COL_GEMM, out_dtype=torch.float32)
    yl = mdnn.conv2d_fwd_algo(X, Wt, pad, mdnn.CONV_IM2COL_GEMM, bias=dev(b, "f32"), act=mdnn.ACT_RELU)
    torch.cuda.synchronize()
    x64, w64 = decode(x, dt), decode(wt, dt)
    exact = ops.conv2d_fwd(x64, w64, pad)
    assert norm_max_err(host64(y32), exact) <= TOL
    exact_b = ops.bias_act(exact, b.astype(np.float64), "relu")
    kk = r * s * ci + 1
    err = accum_bound(ops.conv2d_fwd(np.abs(x64), np.abs(w64), pad) + np.abs(b), kk)
    if dt == "f32":
        err = err * 2.0     # fp32 operands: each product rounds too
        assert np.all(np.abs(host64(yl) - exact_b) <= err)
    else:
        assert lowp_close(host64(yl), exact_b, dt, err)


def test_im2col_gemm_integer_exact(mdnn):
    import torch
    n, h, w, ci, co, r, s, pad = 2, 10, 9, 32, 48, 3, 3, 1
    x = W.small_ints((n, h, w, ci), 72, 1, dtype="f16")
    wt = W.small_ints((co, r, s, ci), 72, 2, dtype="f16")
    y = mdnn.conv2d_fwd_algo(dev(x, "f16"), dev(wt, "f16"), pad, mdnn.CONV_IM2COL_GEMM, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert np.array_equal(host64(y), ops.conv2d_fwd(x.astype(np.float64), wt.astype(np.float64), pad))


@pytest.mark.parametrize("layer", range(3))
def test_im2col_gemm_resnet_full_size(mdnn, layer):
    import torch
    sh = W.RESNET_LAYERS[layer]
    x, wt, _ = W.conv_operands(sh)
    y = mdnn.conv2d_fwd_algo(dev(x, "f16"), dev(wt, "f16"), sh.pad, mdnn.CONV_IM2COL_GEMM, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = ops.conv2d_fwd(x.astype(np.float64), wt.astype(np.float64), sh.pad)
    assert norm_max_err(host64(y), ref) <= TOL


def test_auto_and_explicit_dispatch(mdnn):
    """AUTO without workspace and IMPLICIT_GEMM are the implicit GEMM;
    WINOGRAD is the Winograd entry point; each bitwise equal to calling it."""
    import torch
    sh = W.RESNET_LAYERS[1]
    x, wt, _ = W.conv_operands(sh)
    X, Wt = dev(x, "f16"), dev(wt, "f16")
    b = dev(W.normal((sh.c_out,), 73, 1, "f32", 0.1), "f32")
    ref = mdnn.conv2d_fwd(X, Wt, sh.pad, bias=b, act=mdnn.ACT_RELU)
    cs = mdnn.ConvShape(sh.n, sh.h, sh.w, sh.c_in, sh.c_out, sh.r, sh.s, sh.pad)
    assert mdnn.mdnn_conv2d_fwd_choose(cs, mdnn.F16, 0) == mdnn.CONV_IMPLICIT_GEMM
    for algo in (mdnn.CONV_AUTO, mdnn.CONV_IMPLICIT_GEMM):
        y = torch.empty_like(ref)
        mdnn.mdnn_conv2d_fwd_algo(cs, X, Wt, mdnn.F16, b, mdnn.ACT_RELU, y, mdnn.F16, algo, None, 0)
        torch.cuda.synchronize()
        assert torch.equal(y, ref)
    wino = mdnn.conv2d_fwd_winograd(X, Wt, sh.pad, bias=b, act=mdnn.ACT_RELU)
    via = mdnn.conv2d_fwd_algo(X, Wt, sh.pad, mdnn.CONV_WINOGRAD, bias=b, act=mdnn.ACT_RELU)
    torch.cuda.synchronize()
    assert torch.equal(wino, via)
    # AUTO with room for every algorithm: whichever the table picks, the
    # result keeps the implicit GEMM's accuracy (never Winograd)
    ws = max(mdnn.mdnn_conv2d_fwd_algo_workspace(cs, mdnn.F16, a) for a in (2, 3))
    algo = mdnn.mdnn_conv2d_fwd_choose(cs, mdnn.F16, ws)
    assert algo in (mdnn.CONV_IMPLICIT_GEMM, mdnn.CONV_IM2COL_GEMM)
