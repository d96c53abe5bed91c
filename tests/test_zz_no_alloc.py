"""mdnn_conv2d_bwd_filter_noalloc: the filter gradient with its workspace in
a fixed per-GPU device array instead of a caller buffer (for callers that
cannot allocate).  Called through the C ABI twice in a row, the second call
with a smaller input, and compared with mdnn_conv2d_bwd_filter on a caller
workspace: the same kernels run, so dw and db must be bitwise equal; the
small case is also checked against the oracle."""
import numpy as np
import pytest

import workloads as W
from oracle import ops
from oracle.rounding import decode
from tests.helpers import dev, host64, norm_max_err

pytestmark = pytest.mark.gpu


def _reference(mdnn, cs, X, DY, io, dw_shape):
    import torch
    need = mdnn.mdnn_conv2d_bwd_filter_workspace(cs, io)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device="cuda")
    dw = torch.empty(dw_shape, dtype=torch.float32, device="cuda")
    db = torch.empty((dw_shape[0],), dtype=torch.float32, device="cuda")
    mdnn.mdnn_conv2d_bwd_filter(cs, X, DY, io, dw, db, ws, need)
    return dw, db


def _noalloc(mdnn, cs, X, DY, io, dw_shape):
    import torch
    dw = torch.full(dw_shape, float("nan"), dtype=torch.float32, device="cuda")
    db = torch.full((dw_shape[0],), float("nan"), dtype=torch.float32, device="cuda")
    mdnn.mdnn_conv2d_bwd_filter_noalloc(cs, X, DY, io, dw, db)
    return dw, db


def test_noalloc_bwd_filter_matches_workspace_entry_twice(mdnn):
    import torch
    limit = mdnn.mdnn_conv2d_bwd_filter_noalloc_max_workspace()
    assert limit == 48 << 20
    # call 1: the largest ResNet-style layer (its workspace is most of the array)
    sh = W.RESNET_LAYERS[2]
    cs = mdnn.ConvShape(sh.n, sh.h, sh.w, sh.c_in, sh.c_out, sh.r, sh.s, sh.pad)
    assert 16 << 20 < mdnn.mdnn_conv2d_bwd_filter_workspace(cs, mdnn.F16) <= limit
    x, wt, dy = W.conv_operands(sh)
    X, DY = dev(x, "f16"), dev(dy, "f16")
    got = _noalloc(mdnn, cs, X, DY, mdnn.F16, tuple(wt.shape))
    ref = _reference(mdnn, cs, X, DY, mdnn.F16, tuple(wt.shape))
    torch.cuda.synchronize()
    assert torch.equal(got[0], ref[0]) and torch.equal(got[1], ref[1])

    # call 2: a smaller, ragged bf16 input on the same array
    n, h, w, ci, co, r, s, pad = 5, 9, 7, 32, 48, 3, 3, 1
    cs2 = mdnn.ConvShape(n, h, w, ci, co, r, s, pad)
    assert 0 < mdnn.mdnn_conv2d_bwd_filter_workspace(cs2, mdnn.BF16) < mdnn.mdnn_conv2d_bwd_filter_workspace(cs, mdnn.F16)
    x2 = W.normal((n, h, w, ci), 61, 1, "bf16", 0.5)
    dy2 = W.normal((n, h, w, co), 61, 2, "bf16", 0.5)
    X2, DY2 = dev(x2, "bf16"), dev(dy2, "bf16")
    got2 = _noalloc(mdnn, cs2, X2, DY2, mdnn.BF16, (co, r, s, ci))
    ref2 = _reference(mdnn, cs2, X2, DY2, mdnn.BF16, (co, r, s, ci))
    torch.cuda.synchronize()
    assert torch.equal(got2[0], ref2[0]) and torch.equal(got2[1], ref2[1])
    x64, dy64 = decode(x2, "bf16"), decode(dy2, "bf16")
    assert norm_max_err(host64(got2[0]), ops.conv2d_bwd_filter(x64, dy64, pad, r, s)) <= 1e-4
    assert norm_max_err(host64(got2[1]), dy64.sum(axis=(0, 1, 2))) <= 1e-4
