"""GPU parity of the 3x3 halo convolutions (64 channels in the convolved
tensor, its tile and border staged in LDS): forward and backward data
against the oracle's direct definitions, with the filter and bias gradients
of the same layers (the implicit GEMM).

Shapes cover each way a workgroup's 256 output pixels fall on the image:
eight rows of a 32-wide image, one whole 16x16 image, four whole 8x8 images,
and rows of a non-square image; output channels 64 and 128 (one and two
workgroup columns) in each direction (a shape whose forward pass has 64
input channels runs its backward data on the implicit GEMM unless c_out is
64 too, and the other way round).  Small integers make every product and
partial sum exact in fp32, so the fp32 outputs must match the oracle bit for
bit (padding zeros included); the bias + ReLU and mask epilogues stored in
16 bits are checked within one ulp plus the accumulation bound; and the same
layer through the implicit GEMM's pipelined kernels (forced with the
pipelined tile code) agrees with the oracle too.
"""
import numpy as np
import pytest

import workloads as W
from oracle import ops
from oracle.rounding import decode
from tests.helpers import accum_bound, dev, host64, lowp_close, norm_max_err

pytestmark = pytest.mark.gpu

HALO = [  # n, h, w, c_in, c_out
    (2, 32, 32, 64, 64),    # forward and backward data
    (3, 16, 16, 64, 128),   # forward
    (3, 16, 16, 128, 64),   # backward data
    (8, 8, 8, 64, 128),     # forward
    (8, 8, 8, 128, 64),     # backward data
    (1, 16, 32, 64, 64),    # forward and backward data
    (3, 16, 16, 64, 64),    # forward and backward data
]


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("shape", HALO)
def test_halo_integer_exact(mdnn, shape, dt):
    import torch
    n, h, w, ci, co = shape
    x = W.small_ints((n, h, w, ci), 23, 1, dtype=dt)
    wt = W.small_ints((co, 3, 3, ci), 23, 2, dtype=dt)
    dy = W.small_ints((n, h, w, co), 23, 3, dtype=dt)
    X, Wt, DY = dev(x, dt), dev(wt, dt), dev(dy, dt)
    y = mdnn.conv2d_fwd(X, Wt, 1, out_dtype=torch.float32)
    dx = mdnn.conv2d_bwd_data(DY, Wt, 1, h, w, out_dtype=torch.float32)
    dwt, db = mdnn.conv2d_bwd_filter(X, DY, 3, 3, 1)
    torch.cuda.synchronize()
    x64, w64, dy64 = decode(x, dt), decode(wt, dt), decode(dy, dt)
    assert np.array_equal(host64(y), ops.conv2d_fwd(x64, w64, 1))
    assert np.array_equal(host64(dx), ops.conv2d_bwd_data(dy64, w64, 1, h, w))
    assert np.array_equal(host64(dwt), ops.conv2d_bwd_filter(x64, dy64, 1, 3, 3))
    assert np.array_equal(host64(db), dy64.sum(axis=(0, 1, 2)))


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("shape", [HALO[0], HALO[4]])
def test_halo_bias_relu_and_mask_lowp(mdnn, shape, dt):
    """Forward with bias + ReLU stored in the storage type; backward data with
    the ReLU mask of the layer input, stored in the storage type."""
    import torch
    n, h, w, ci, co = shape
    x = W.normal((n, h, w, ci), 24, 1, dt, 0.3)
    wt = W.normal((co, 3, 3, ci), 24, 2, dt, 1 / np.sqrt(9 * ci))
    b = W.normal((co,), 24, 3, "f32", 0.2)
    dy = W.normal((n, h, w, co), 24, 4, dt)
    X, Wt = dev(x, dt), dev(wt, dt)
    y = mdnn.conv2d_fwd(X, Wt, 1, bias=dev(b, "f32"), act=mdnn.ACT_RELU)
    dx = mdnn.conv2d_bwd_data(dev(dy, dt), Wt, 1, h, w, mask=X)
    torch.cuda.synchronize()
    x64, w64, dy64 = decode(x, dt), decode(wt, dt), decode(dy, dt)
    exact = ops.bias_act(ops.conv2d_fwd(x64, w64, 1), b.astype(np.float64), "relu")
    err = accum_bound(ops.conv2d_fwd(np.abs(x64), np.abs(w64), 1) + np.abs(b), 9 * ci + 1)
    assert lowp_close(host64(y), exact, dt, err)
    exact_dx = np.where(x64 > 0, ops.conv2d_bwd_data(dy64, w64, 1, h, w), 0.0)
    err = accum_bound(ops.conv2d_bwd_data(np.abs(dy64), np.abs(w64), 1, h, w), 9 * co)
    assert lowp_close(host64(dx), exact_dx, dt, err)


@pytest.mark.parametrize("tile", [0, 4])
def test_halo_and_implicit_gemm_against_oracle(mdnn, tile):
    """Tile code 0 takes the halo kernels, 4 forces the implicit GEMM's
    pipelined kernels on the same layer: both within 1e-4 of the oracle."""
    import torch
    n, h, w, ci, co = HALO[0]
    x = W.normal((n, h, w, ci), 25, 1, "f16", 1 / np.sqrt(9 * ci))
    wt = W.normal((co, 3, 3, ci), 25, 2, "f16", 1 / np.sqrt(9 * ci))
    dy = W.normal((n, h, w, co), 25, 3, "f16")
    mdnn.mdnn_set_gemm_tile(tile)
    try:
        y = mdnn.conv2d_fwd(dev(x, "f16"), dev(wt, "f16"), 1, out_dtype=torch.float32)
        dx = mdnn.conv2d_bwd_data(dev(dy, "f16"), dev(wt, "f16"), 1, h, w, out_dtype=torch.float32)
        torch.cuda.synchronize()
    finally:
        mdnn.mdnn_set_gemm_tile(0)
    x64, w64, dy64 = decode(x, "f16"), decode(wt, "f16"), decode(dy, "f16")
    assert norm_max_err(host64(y), ops.conv2d_fwd(x64, w64, 1)) <= 1e-4
    assert norm_max_err(host64(dx), ops.conv2d_bwd_data(dy64, w64, 1, h, w)) <= 1e-4
