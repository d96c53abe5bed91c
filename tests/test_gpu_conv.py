"""GPU parity of the implicit-GEMM convolutions against the oracle's direct
definitions (fwd, bwd-data, bwd-filter; stride 1, zero padding, NHWC x KRSC).

fp32 outputs: normalized max error <= 1e-4.  Low-precision outputs (with the
bias+ReLU epilogue or the ReLU mask): one storage ulp plus the fp32
accumulation bound.  Covers channel counts that are and are not multiples of
8 (vector and element-wise operand paths), the pipelined kernels (c_in or
c_out multiples of 64) next to the general ones, non-"same" padding, the LeNet-style
layers (Cin = 1 and 32, 5x5) and the three ResNet-style 3x3 layers at their
full size (batch 128), as launched by the benchmark.
"""
import numpy as np
import pytest

import workloads as W
from oracle import ops
from oracle.rounding import decode
from tests.helpers import DT, accum_bound, dev, host64, lowp_close, norm_max_err

pytestmark = pytest.mark.gpu
TOL = 1e-4

SMALL = [  # n, h, w, c_in, c_out, r, s, pad
    (2, 5, 4, 8, 16, 3, 3, 1),
    (2, 7, 6, 3, 5, 3, 3, 1),
    (1, 6, 6, 1, 32, 5, 5, 2),
    (3, 9, 9, 16, 24, 3, 3, 0),
    (2, 6, 7, 24, 8, 5, 3, 2),
    (2, 14, 14, 32, 64, 5, 5, 2),
    (1, 3, 3, 8, 8, 5, 5, 1),
]


def _ops(mdnn, shape, dt, seed):
    import torch
    n, h, w, ci, co, r, s, pad = shape
    ho, wo = h + 2 * pad - r + 1, w + 2 * pad - s + 1
    x = W.normal((n, h, w, ci), seed, 1, dt, 1 / np.sqrt(r * s * ci))
    wt = W.normal((co, r, s, ci), seed, 2, dt, 1 / np.sqrt(r * s * ci))
    dy = W.normal((n, ho, wo, co), seed, 3, dt, 1 / np.sqrt(r * s * ci))
    X, Wt, DY = dev(x, dt), dev(wt, dt), dev(dy, dt)
    y = mdnn.conv2d_fwd(X, Wt, pad, out_dtype=torch.float32)
    dx = mdnn.conv2d_bwd_data(DY, Wt, pad, h, w, out_dtype=torch.float32)
    dwt, db = mdnn.conv2d_bwd_filter(X, DY, r, s, pad)
    torch.cuda.synchronize()
    return (decode(x, dt), decode(wt, dt), decode(dy, dt)), (host64(y), host64(dx), host64(dwt), host64(db))


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("shape", SMALL)
def test_conv_small_against_oracle(mdnn, shape, dt):
    n, h, w, ci, co, r, s, pad = shape
    (x, wt, dy), (y, dx, dw, db) = _ops(mdnn, shape, dt, 11)
    assert norm_max_err(y, ops.conv2d_fwd(x, wt, pad)) <= TOL
    assert norm_max_err(dx, ops.conv2d_bwd_data(dy, wt, pad, h, w)) <= TOL
    assert norm_max_err(dw, ops.conv2d_bwd_filter(x, dy, pad, r, s)) <= TOL
    assert norm_max_err(db, dy.sum(axis=(0, 1, 2))) <= TOL


# Shapes on the direct small-reduction kernels (r*s*c_in <= 64; the filter
# gradient also needs c_out*r*s*c_in <= 1024): ragged channel groups,
# valid (non-"same") padding, several 512-pixel filter blocks with a ragged
# tail, the largest filter gradient (1024 outputs), c_out = 256 (forward
# only: its filter gradient exceeds the LDS budget and takes the GEMM path).
DIRECT = [  # n, h, w, c_in, c_out, r, s, pad
    (3, 13, 11, 3, 10, 3, 3, 1),
    (2, 9, 8, 2, 7, 3, 3, 0),
    (5, 17, 15, 1, 32, 5, 5, 2),
    (2, 10, 9, 4, 16, 4, 4, 1),
    (2, 6, 5, 3, 256, 1, 1, 0),
    (1, 1, 1, 64, 4, 1, 1, 0),
]


@pytest.mark.parametrize("dt", ["f16", "bf16", "f32"])
@pytest.mark.parametrize("shape", DIRECT)
def test_conv_direct_against_oracle(mdnn, shape, dt):
    n, h, w, ci, co, r, s, pad = shape
    (x, wt, dy), (y, dx, dw, db) = _ops(mdnn, shape, dt, 23)
    assert norm_max_err(y, ops.conv2d_fwd(x, wt, pad)) <= TOL
    assert norm_max_err(dx, ops.conv2d_bwd_data(dy, wt, pad, h, w)) <= TOL
    assert norm_max_err(dw, ops.conv2d_bwd_filter(x, dy, pad, r, s)) <= TOL
    assert norm_max_err(db, dy.sum(axis=(0, 1, 2))) <= TOL


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_conv_direct_epilogue_lowp(mdnn, dt):
    """Direct forward with bias+ReLU stored in the storage type (c_out = 10:
    a ragged group of four channels), ragged pixel count."""
    n, h, w, ci, co, r, s, pad = 3, 7, 9, 2, 10, 5, 5, 2
    x = W.normal((n, h, w, ci), 24, 1, dt, 0.3)
    wt = W.normal((co, r, s, ci), 24, 2, dt, 0.3)
    b = W.normal((co,), 24, 3, "f32", 0.2)
    y = mdnn.conv2d_fwd(dev(x, dt), dev(wt, dt), pad, bias=dev(b, "f32"), act=mdnn.ACT_RELU)
    x64, w64 = decode(x, dt), decode(wt, dt)
    exact = ops.bias_act(ops.conv2d_fwd(x64, w64, pad), b.astype(np.float64), "relu")
    err = accum_bound(ops.conv2d_fwd(np.abs(x64), np.abs(w64), pad) + np.abs(b), r * s * ci + 1)
    assert lowp_close(host64(y), exact, dt, err)


def test_conv_direct_integer_exact(mdnn):
    import torch
    n, h, w, ci, co, r, s, pad = 4, 12, 11, 2, 12, 5, 5, 2
    x = W.small_ints((n, h, w, ci), 25, 1, dtype="f16")
    wt = W.small_ints((co, r, s, ci), 25, 2, dtype="f16")
    dy = W.small_ints((n, h, w, co), 25, 3, dtype="f16")
    X, Wt, DY = dev(x, "f16"), dev(wt, "f16"), dev(dy, "f16")
    y = mdnn.conv2d_fwd(X, Wt, pad, out_dtype=torch.float32)
    dwt, _ = mdnn.conv2d_bwd_filter(X, DY, r, s, pad)
    torch.cuda.synchronize()
    x64, w64, dy64 = x.astype(np.float64), wt.astype(np.float64), dy.astype(np.float64)
    assert np.array_equal(host64(y), ops.conv2d_fwd(x64, w64, pad))
    assert np.array_equal(host64(dwt), ops.conv2d_bwd_filter(x64, dy64, pad, r, s))


# Shapes on the pipelined kernels (forward: c_in % 64 == 0; backward data:
# c_out % 64 == 0 and c_in % 8 == 0; backward filter: size-preserving, channels
# multiples of 8, n*h*w % 64 == 0), with ragged M and N, non-square grids,
# padding that changes the output size, 1x1 and 5x5 taps and split-K.
PIPE = [  # n, h, w, c_in, c_out, r, s, pad
    (2, 7, 9, 64, 72, 3, 3, 1),      # fwd, N = 72 (128 x 128 tile, ragged)
    (3, 5, 6, 128, 64, 3, 3, 0),     # fwd + bwd_data with ho != h (valid conv)
    (2, 8, 8, 64, 128, 5, 5, 2),     # all three; filter single split
    (4, 16, 16, 64, 64, 1, 1, 0),    # 1x1; filter split-K on the 64-row tile
    (2, 12, 10, 192, 40, 3, 3, 1),   # fwd, N = 40 (256 x 64 tile)
    (5, 11, 13, 64, 64, 3, 3, 1),    # ragged M = 715
    (8, 16, 16, 64, 256, 3, 3, 1),   # filter split-K on the 128 x 128 tile
    (2, 8, 8, 16, 8, 3, 3, 1),       # filter with c_out = 8
]


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("shape", PIPE)
def test_conv_pipelined_against_oracle(mdnn, shape, dt):
    n, h, w, ci, co, r, s, pad = shape
    (x, wt, dy), (y, dx, dw, db) = _ops(mdnn, shape, dt, 17)
    assert norm_max_err(y, ops.conv2d_fwd(x, wt, pad)) <= TOL
    assert norm_max_err(dx, ops.conv2d_bwd_data(dy, wt, pad, h, w)) <= TOL
    assert norm_max_err(dw, ops.conv2d_bwd_filter(x, dy, pad, r, s)) <= TOL
    assert norm_max_err(db, dy.sum(axis=(0, 1, 2))) <= TOL


# Forward on the pipelined kernel with c_in a multiple of 32 but not of 64:
# two 32-channel half blocks per K step, the K range padded to whole steps
# (odd half-block counts: 3x3, 1x1, 5x3 taps at c_in = 32), several half
# blocks per tap (c_in = 96, 160), both tile shapes, ragged M, valid and
# wider padding.
PIPE32 = [  # n, h, w, c_in, c_out, r, s, pad
    (2, 14, 14, 32, 64, 5, 5, 2),    # LeNet conv2 shape at batch 2 (25 taps: a padded half block)
    (3, 7, 9, 32, 40, 3, 3, 1),      # 9 taps, 256 x 64 tile, ragged M = 189
    (2, 6, 5, 32, 72, 1, 1, 0),      # 1x1: one real half block per step, 128 x 128 tile
    (2, 9, 7, 96, 24, 3, 3, 0),      # three half blocks per tap, valid padding
    (1, 8, 11, 160, 136, 5, 3, 2),   # five half blocks per tap, 5x3 taps, N = 136
]


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("shape", PIPE32)
def test_conv_fwd_32_channel_blocks_against_oracle(mdnn, shape, dt):
    n, h, w, ci, co, r, s, pad = shape
    (x, wt, dy), (y, dx, dw, db) = _ops(mdnn, shape, dt, 23)
    assert norm_max_err(y, ops.conv2d_fwd(x, wt, pad)) <= TOL
    assert norm_max_err(dx, ops.conv2d_bwd_data(dy, wt, pad, h, w)) <= TOL
    assert norm_max_err(dw, ops.conv2d_bwd_filter(x, dy, pad, r, s)) <= TOL


def test_conv_fwd_32_channel_blocks_epilogue_and_integers(mdnn):
    """The same path with bias + ReLU into bf16 (bound as for the other
    pipelined forward), and bit-exact on small integers (the padded half
    block contributes exact zeros)."""
    import torch
    n, h, w, ci, co, r, s, pad = 3, 9, 7, 32, 48, 3, 3, 1
    x = W.normal((n, h, w, ci), 24, 1, "bf16", 0.3)
    wt = W.normal((co, r, s, ci), 24, 2, "bf16", 0.1)
    b = W.normal((co,), 24, 3, "f32", 0.2)
    y = mdnn.conv2d_fwd(dev(x, "bf16"), dev(wt, "bf16"), pad, bias=dev(b, "f32"), act=mdnn.ACT_RELU)
    torch.cuda.synchronize()
    x64, w64 = decode(x, "bf16"), decode(wt, "bf16")
    exact = ops.bias_act(ops.conv2d_fwd(x64, w64, pad), b.astype(np.float64), "relu")
    err = accum_bound(ops.conv2d_fwd(np.abs(x64), np.abs(w64), pad) + np.abs(b), r * s * ci + 1)
    assert lowp_close(host64(y), exact, "bf16", err)
    xi = W.small_ints((n, h, w, ci), 25, 1, dtype="f16")
    wi = W.small_ints((co, r, s, ci), 25, 2, dtype="f16")
    yi = mdnn.conv2d_fwd(dev(xi, "f16"), dev(wi, "f16"), pad, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert np.array_equal(host64(yi), ops.conv2d_fwd(xi.astype(np.float64), wi.astype(np.float64), pad))


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_conv_pipelined_epilogues_lowp(mdnn, dt):
    """Pipelined forward with bias+ReLU stored in the storage type, pipelined
    backward-data with the ReLU mask, both with ragged M."""
    import torch
    n, h, w, ci, co, r, s, pad = 3, 7, 5, 64, 64, 3, 3, 1
    x = W.normal((n, h, w, ci), 18, 1, dt, 0.3)
    wt = W.normal((co, r, s, ci), 18, 2, dt, 0.1)
    b = W.normal((co,), 18, 3, "f32", 0.2)
    dy = W.normal((n, h, w, co), 18, 4, dt)
    X, Wt = dev(x, dt), dev(wt, dt)
    y = mdnn.conv2d_fwd(X, Wt, pad, bias=dev(b, "f32"), act=mdnn.ACT_RELU)
    dx = mdnn.conv2d_bwd_data(dev(dy, dt), Wt, pad, h, w, mask=X)
    torch.cuda.synchronize()
    x64, w64, dy64 = decode(x, dt), decode(wt, dt), decode(dy, dt)
    exact = ops.bias_act(ops.conv2d_fwd(x64, w64, pad), b.astype(np.float64), "relu")
    err = accum_bound(ops.conv2d_fwd(np.abs(x64), np.abs(w64), pad) + np.abs(b), r * s * ci + 1)
    assert lowp_close(host64(y), exact, dt, err)
    exact_dx = np.where(x64 > 0, ops.conv2d_bwd_data(dy64, w64, pad, h, w), 0.0)
    err = accum_bound(ops.conv2d_bwd_data(np.abs(dy64), np.abs(w64), pad, h, w), r * s * co)
    assert lowp_close(host64(dx), exact_dx, dt, err)


def test_conv_pipelined_integer_exact(mdnn):
    """Small integers: every product and partial sum is exact in fp32, so the
    pipelined kernels (padding zeros included) must match bit for bit."""
    import torch
    n, h, w, ci, co, r, s, pad = 2, 8, 8, 64, 64, 3, 3, 1
    x = W.small_ints((n, h, w, ci), 19, 1, dtype="f16")
    wt = W.small_ints((co, r, s, ci), 19, 2, dtype="f16")
    dy = W.small_ints((n, h, w, co), 19, 3, dtype="f16")
    X, Wt, DY = dev(x, "f16"), dev(wt, "f16"), dev(dy, "f16")
    y = mdnn.conv2d_fwd(X, Wt, pad, out_dtype=torch.float32)
    dx = mdnn.conv2d_bwd_data(DY, Wt, pad, h, w, out_dtype=torch.float32)
    dwt, db = mdnn.conv2d_bwd_filter(X, DY, r, s, pad)
    torch.cuda.synchronize()
    x64, w64, dy64 = x.astype(np.float64), wt.astype(np.float64), dy.astype(np.float64)
    assert np.array_equal(host64(y), ops.conv2d_fwd(x64, w64, pad))
    assert np.array_equal(host64(dx), ops.conv2d_bwd_data(dy64, w64, pad, h, w))
    assert np.array_equal(host64(dwt), ops.conv2d_bwd_filter(x64, dy64, pad, r, s))


@pytest.mark.parametrize("tile", [1, 2, 3])
def test_conv_all_tiles(mdnn, tile):
    mdnn.mdnn_set_gemm_tile(tile)
    try:
        shape = (2, 9, 7, 16, 24, 3, 3, 1)
        n, h, w, ci, co, r, s, pad = shape
        (x, wt, dy), (y, dx, dw, db) = _ops(mdnn, shape, "f16", 12)
        assert norm_max_err(y, ops.conv2d_fwd(x, wt, pad)) <= TOL
        assert norm_max_err(dx, ops.conv2d_bwd_data(dy, wt, pad, h, w)) <= TOL
        assert norm_max_err(dw, ops.conv2d_bwd_filter(x, dy, pad, r, s)) <= TOL
    finally:
        mdnn.mdnn_set_gemm_tile(0)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_conv_bias_relu_and_mask_lowp(mdnn, dt):
    """Forward with bias+ReLU stored in the storage type; backward-data with
    the ReLU mask of the layer input, stored in the storage type."""
    import torch
    n, h, w, ci, co, r, s, pad = 2, 8, 8, 16, 32, 3, 3, 1
    x = W.normal((n, h, w, ci), 13, 1, dt, 0.3)
    wt = W.normal((co, r, s, ci), 13, 2, dt, 0.3)
    b = W.normal((co,), 13, 3, "f32", 0.2)
    dy = W.normal((n, h, w, co), 13, 4, dt)
    X, Wt = dev(x, dt), dev(wt, dt)
    y = mdnn.conv2d_fwd(X, Wt, pad, bias=dev(b, "f32"), act=mdnn.ACT_RELU)
    dx = mdnn.conv2d_bwd_data(dev(dy, dt), Wt, pad, h, w, mask=X)
    torch.cuda.synchronize()
    x64, w64, dy64 = decode(x, dt), decode(wt, dt), decode(dy, dt)
    exact = ops.bias_act(ops.conv2d_fwd(x64, w64, pad), b.astype(np.float64), "relu")
    err = accum_bound(ops.conv2d_fwd(np.abs(x64), np.abs(w64), pad) + np.abs(b), r * s * ci + 1)
    assert lowp_close(host64(y), exact, dt, err)
    exact_dx = np.where(x64 > 0, ops.conv2d_bwd_data(dy64, w64, pad, h, w), 0.0)
    err = accum_bound(ops.conv2d_bwd_data(np.abs(dy64), np.abs(w64), pad, h, w), r * s * co)
    assert lowp_close(host64(dx), exact_dx, dt, err)


def test_conv_integer_exact(mdnn):
    import torch
    n, h, w, ci, co, r, s, pad = 2, 10, 10, 16, 16, 3, 3, 1
    x = W.small_ints((n, h, w, ci), 14, 1, dtype="f16")
    wt = W.small_ints((co, r, s, ci), 14, 2, dtype="f16")
    dy = W.small_ints((n, h, w, co), 14, 3, dtype="f16")
    X, Wt, DY = dev(x, "f16"), dev(wt, "f16"), dev(dy, "f16")
    y = mdnn.conv2d_fwd(X, Wt, pad, out_dtype=torch.float32)
    dx = mdnn.conv2d_bwd_data(DY, Wt, pad, h, w, out_dtype=torch.float32)
    dwt, db = mdnn.conv2d_bwd_filter(X, DY, r, s, pad)
    torch.cuda.synchronize()
    x64, w64, dy64 = x.astype(np.float64), wt.astype(np.float64), dy.astype(np.float64)
    assert np.array_equal(host64(y), ops.conv2d_fwd(x64, w64, pad))
    assert np.array_equal(host64(dx), ops.conv2d_bwd_data(dy64, w64, pad, h, w))
    assert np.array_equal(host64(dwt), ops.conv2d_bwd_filter(x64, dy64, pad, r, s))


def test_conv_fp32_path(mdnn):
    shape = (2, 6, 5, 3, 4, 3, 3, 1)
    n, h, w, ci, co, r, s, pad = shape
    (x, wt, dy), (y, dx, dw, db) = _ops(mdnn, shape, "f32", 15)
    assert norm_max_err(y, ops.conv2d_fwd(x, wt, pad)) <= 1e-6
    assert norm_max_err(dx, ops.conv2d_bwd_data(dy, wt, pad, h, w)) <= 1e-6
    assert norm_max_err(dw, ops.conv2d_bwd_filter(x, dy, pad, r, s)) <= 1e-6


@pytest.mark.parametrize("layer", range(3))
def test_resnet_layers_full_size(mdnn, layer):
    """The ResNet-style 3x3 layers at batch 128 (fp16 in, fp32 out): all three
    operations against the full oracle."""
    import torch
    sh = W.RESNET_LAYERS[layer]
    x, wt, dy = W.conv_operands(sh)
    X, Wt, DY = dev(x, "f16"), dev(wt, "f16"), dev(dy, "f16")
    y = mdnn.conv2d_fwd(X, Wt, sh.pad, out_dtype=torch.float32)
    dx = mdnn.conv2d_bwd_data(DY, Wt, sh.pad, sh.h, sh.w, out_dtype=torch.float32)
    dwt, db = mdnn.conv2d_bwd_filter(X, DY, sh.r, sh.s, sh.pad)
    torch.cuda.synchronize()
    x64, w64, dy64 = x.astype(np.float64), wt.astype(np.float64), dy.astype(np.float64)
    assert norm_max_err(host64(y), ops.conv2d_fwd(x64, w64, sh.pad)) <= TOL
    assert norm_max_err(host64(dx), ops.conv2d_bwd_data(dy64, w64, sh.pad, sh.h, sh.w)) <= TOL
    assert norm_max_err(host64(dwt), ops.conv2d_bwd_filter(x64, dy64, sh.pad, sh.r, sh.s)) <= TOL
    assert norm_max_err(host64(db), dy64.sum(axis=(0, 1, 2))) <= TOL


@pytest.mark.parametrize("layer", range(3))
def test_resnet_layers_full_size_fp16_out(mdnn, layer):
    """The same layers with fp16 outputs, the instantiations the benchmark
    times: each stored value is the fp16 rounding of a value within the fp32
    accumulation bound of the exact convolution (one fp16 rounding alone
    exceeds 1e-4 of the maximum, so the bar is one ulp plus that bound)."""
    import torch
    sh = W.RESNET_LAYERS[layer]
    x, wt, dy = W.conv_operands(sh)
    X, Wt, DY = dev(x, "f16"), dev(wt, "f16"), dev(dy, "f16")
    y = mdnn.conv2d_fwd(X, Wt, sh.pad)
    dx = mdnn.conv2d_bwd_data(DY, Wt, sh.pad, sh.h, sh.w)
    torch.cuda.synchronize()
    assert y.dtype == torch.float16 and dx.dtype == torch.float16
    x64, w64, dy64 = x.astype(np.float64), wt.astype(np.float64), dy.astype(np.float64)
    kk = sh.r * sh.s * sh.c_in
    err = accum_bound(ops.conv2d_fwd(np.abs(x64), np.abs(w64), sh.pad), kk)
    assert lowp_close(host64(y), ops.conv2d_fwd(x64, w64, sh.pad), "f16", err)
    err = accum_bound(ops.conv2d_bwd_data(np.abs(dy64), np.abs(w64), sh.pad, sh.h, sh.w), kk)
    assert lowp_close(host64(dx), ops.conv2d_bwd_data(dy64, w64, sh.pad, sh.h, sh.w), "f16", err)


@pytest.mark.parametrize("which", ["conv1", "conv2"])
def test_lenet_conv_layers(mdnn, which):
    """LeNet-style convolutions at batch 256 in bf16 (conv1: Cin = 1, the
    element-wise operand path; conv2: Cin = 32), fp32 outputs."""
    import torch
    ci, co, h = (1, 32, 28) if which == "conv1" else (32, 64, 14)
    n, r, pad = 256, 5, 2
    x = W.normal((n, h, h, ci), 16, 1, "bf16", 0.5)
    wt = W.normal((co, r, r, ci), 16, 2, "bf16", np.sqrt(2 / (25 * ci)))
    dy = W.normal((n, h, h, co), 16, 3, "bf16", 1e-3)
    X, Wt, DY = dev(x, "bf16"), dev(wt, "bf16"), dev(dy, "bf16")
    y = mdnn.conv2d_fwd(X, Wt, pad, out_dtype=torch.float32)
    dwt, db = mdnn.conv2d_bwd_filter(X, DY, r, r, pad)
    dx = mdnn.conv2d_bwd_data(DY, Wt, pad, h, h, out_dtype=torch.float32)
    torch.cuda.synchronize()
    x64, w64, dy64 = decode(x, "bf16"), decode(wt, "bf16"), decode(dy, "bf16")
    assert norm_max_err(host64(y), ops.conv2d_fwd(x64, w64, pad)) <= TOL
    assert norm_max_err(host64(dwt), ops.conv2d_bwd_filter(x64, dy64, pad, r, r)) <= TOL
    assert norm_max_err(host64(dx), ops.conv2d_bwd_data(dy64, w64, pad, h, h)) <= TOL


def test_conv_bwd_filter_deterministic(mdnn):
    """Split-K partials are reduced in a fixed order: reruns are bitwise equal."""
    import torch
    sh = W.RESNET_LAYERS[0]
    x, wt, dy = W.conv_operands(sh)
    X, DY = dev(x, "f16"), dev(dy, "f16")
    a, _ = mdnn.conv2d_bwd_filter(X, DY, 3, 3, 1)
    b, _ = mdnn.conv2d_bwd_filter(X, DY, 3, 3, 1)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    del wt


@pytest.mark.parametrize("layer", [0, 1])
def test_conv_bwd_filter_batched_sums_bitwise(mdnn, layer):
    """With db the weight and bias sums' second passes share one launch
    (several reductions per grid); without db the weight sums run alone: the
    same sums in the same order, so dw is bitwise the same, and db is
    deterministic too."""
    import torch
    sh = W.RESNET_LAYERS[layer]
    x, wt, dy = W.conv_operands(sh)
    X, DY = dev(x, "f16"), dev(dy, "f16")
    a, db1 = mdnn.conv2d_bwd_filter(X, DY, 3, 3, 1)
    b, _ = mdnn.conv2d_bwd_filter(X, DY, 3, 3, 1, with_db=False)
    c, db2 = mdnn.conv2d_bwd_filter(X, DY, 3, 3, 1)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    assert torch.equal(a.view(torch.int32), c.view(torch.int32))
    assert torch.equal(db1.view(torch.int32), db2.view(torch.int32))
    del wt
