"""GPU parity of the Winograd F(2x2, 3x3) forward convolution (section 2.1's
swappable convolution algorithm) against the convolution's plain definition
(ops.conv2d_fwd).

The algorithm rounds its transformed operands U = G g G^T and V = B^T d B
once to the storage type before the matrix-core products, so its error bar is
derived from that arithmetic rather than the implicit GEMM's 1e-4: with u the
storage format's unit roundoff,

    |y - conv(x, w)| <= (2u + u^2 + (gamma_C + gamma_16)(1 + u)^2 + gamma_9) * S,
    S = |A^T| (sum_c |U| |V|) |A|             (oracle/winograd.error_scale)

(two operand roundings, the fp32 sum over C channels, the fp32 transforms).
The numpy emulation of this arithmetic in tests/test_oracle_winograd.py stays
inside the same bound.  Low-precision outputs add one storage rounding.
Small integers are exact (all transformed values are multiples of 1/4).
Covers the three ResNet-style layers at full size (batch 128, as the
benchmark runs them), ragged last tiles, valid and wider padding, channel
counts that are not multiples of 8, and the bias + ReLU epilogue.
"""
import numpy as np
import pytest

import workloads as W
from oracle import ops, winograd as wg
from oracle.rounding import decode
from tests.helpers import DT, dev, host64, lowp_close

pytestmark = pytest.mark.gpu

U_FMT = {"f16": 2.0 ** -11, "bf16": 2.0 ** -8}


def _gamma(q):
    return q * 2.0 ** -24 / (1 - q * 2.0 ** -24)


def _coef(dt, c):
    u = U_FMT[dt]
    return 2 * u + u * u + (_gamma(c) + _gamma(16)) * (1 + u) ** 2 + _gamma(9)


def _run(mdnn, x, w, pad, dt, out_dt, bias=None, act=0):
    import torch
    y = mdnn.conv2d_fwd_winograd(dev(x, dt), dev(w, dt), pad, bias=bias, act=act,
                                 out_dtype=torch.float32 if out_dt == "f32" else None)
    torch.cuda.synchronize()
    return host64(y)


@pytest.mark.parametrize("layer", range(3))
def test_resnet_layers_full_size(mdnn, layer):
    sh = W.RESNET_LAYERS[layer]
    x, w, _ = W.conv_operands(sh)
    got = _run(mdnn, x, w, sh.pad, "f16", "f32")
    x64, w64 = x.astype(np.float64), w.astype(np.float64)
    exact = ops.conv2d_fwd(x64, w64, sh.pad)
    bound = _coef("f16", sh.c_in) * wg.error_scale(x64, w64, sh.pad)
    assert np.all(np.abs(got - exact) <= bound)


SHAPES = [  # n, h, w, c_in, c_out, pad
    (2, 7, 9, 16, 24, 1),     # ragged last tiles in both directions
    (3, 8, 8, 64, 64, 1),
    (2, 10, 6, 5, 7, 1),      # channels not multiples of 8 (element loads)
    (1, 9, 9, 8, 72, 0),      # valid padding, c_out > 64
    (2, 5, 5, 24, 16, 2),     # wider padding
    (1, 3, 3, 8, 8, 1),
]


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("shape", SHAPES)
def test_small_shapes_fp32_out(mdnn, dt, shape):
    n, h, wd, c, k, pad = shape
    x = W.normal((n, h, wd, c), 51, 1, dt)
    w = W.normal((k, 3, 3, c), 51, 2, dt, 1 / np.sqrt(9 * c))
    got = _run(mdnn, x, w, pad, dt, "f32")
    x64, w64 = decode(x, dt), decode(w, dt)
    exact = ops.conv2d_fwd(x64, w64, pad)
    assert got.shape == exact.shape
    assert np.all(np.abs(got - exact) <= _coef(dt, c) * wg.error_scale(x64, w64, pad))


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_bias_relu_lowp_out(mdnn, dt):
    n, h, wd, c, k, pad = 2, 9, 7, 32, 20, 1
    x = W.normal((n, h, wd, c), 52, 1, dt)
    w = W.normal((k, 3, 3, c), 52, 2, dt, 1 / np.sqrt(9 * c))
    b = W.normal((k,), 52, 3, "f32", 0.3)
    got = _run(mdnn, x, w, pad, dt, dt, bias=dev(b, "f32"), act=mdnn.ACT_RELU)
    x64, w64 = decode(x, dt), decode(w, dt)
    exact = ops.bias_act(ops.conv2d_fwd(x64, w64, pad), b.astype(np.float64), "relu")
    scale = wg.error_scale(x64, w64, pad)
    err = _coef(dt, c) * scale + 2.0 ** -23 * (scale + np.abs(b))
    assert lowp_close(got, exact, dt, err)
    assert np.all(got >= 0)


def test_small_integers_exact_and_deterministic(mdnn):
    import torch
    n, h, wd, c, k, pad = 2, 11, 10, 16, 24, 1
    x = W.small_ints((n, h, wd, c), 53, 1, lo=-3, hi=3, dtype="f16")
    w = W.small_ints((k, 3, 3, c), 53, 2, lo=-3, hi=3, dtype="f16")
    X, Wt = dev(x, "f16"), dev(w, "f16")
    a = mdnn.conv2d_fwd_winograd(X, Wt, pad, out_dtype=torch.float32)
    b = mdnn.conv2d_fwd_winograd(X, Wt, pad, out_dtype=torch.float32)
    torch.cuda.synchronize()
    want = ops.conv2d_fwd(x.astype(np.float64), w.astype(np.float64), pad)
    assert np.array_equal(host64(a), want)
    assert torch.equal(a, b)
