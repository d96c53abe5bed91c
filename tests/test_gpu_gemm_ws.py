"""GPU parity of mdnn_gemm_mixed_ws (section 3.2's product with a caller
workspace): shapes whose output is a few tiles split K across workgroups into
fp32 partials, summed in a fixed order before the epilogue.

Covers each kernel family that splits: the fp32 kernel, the direct-to-LDS
pipelined kernel (plain 16-byte aligned operands, K % 64 == 0) and the
general MFMA kernel (N = 10, or K not a multiple of 64), in every layout,
with bias + ReLU, beta * C and the ReLU mask.  Bars as for mdnn_gemm_mixed:
fp32 outputs within 1e-4 normalized max error, low-precision outputs within
one storage ulp plus gamma_K * sum |a||b|, small integers bit-exact.  Also:
repeated calls are bitwise equal, and a workspace that is too small (or a
shape that needs no split) gives exactly mdnn_gemm_mixed's result.
"""
import numpy as np
import pytest

import workloads as W
from oracle import ops
from oracle.rounding import decode
from tests.helpers import DT, accum_bound, dev, empty, host64, lowp_close, norm_max_err

pytestmark = pytest.mark.gpu

LAYOUT = {"NN": 0, "NT": 1, "TN": 2}
TOL = 1e-4
SPLIT_SHAPES = [  # (m, n, k): all plan a split
    (256, 1024, 3136),   # 16 tiles of 128 x 128: pipelined kernel
    (256, 10, 1024),     # N = 10: general kernel (fp16 / bf16), fp32 kernel
    (70, 136, 1000),     # K % 64 != 0: general kernel
    (64, 128, 784),
]


def _shapes(layout, m, n, k):
    return ((k, m) if layout == "TN" else (m, k)), ((n, k) if layout == "NT" else (k, n))


def _run(mdnn, layout, A, B, out_dt, m, n, k, ws, bias=None, act=0, mask=None, beta=0.0, Cm=None):
    import torch
    D = empty((m, n), out_dt)
    D.fill_(float("nan"))
    args = (LAYOUT[layout], m, n, k, 1.0, A, A.stride(0), B, B.stride(0), mdnn.dtype_of(A), beta, Cm,
            Cm.stride(0) if Cm is not None else 0, D, D.stride(0), DT[out_dt], bias, act, mask,
            mask.stride(0) if mask is not None else 0)
    if ws is None:
        mdnn.mdnn_gemm_mixed(*args)
    else:
        mdnn.mdnn_gemm_mixed_ws(*args, ws, ws.numel())
    torch.cuda.synchronize()
    return host64(D)


def _ws(mdnn, dt, m, n, k, short=0):
    import torch
    nb = mdnn.mdnn_gemm_workspace(DT[dt], m, n, k)
    return torch.empty((max(nb - short, 16),), dtype=torch.uint8, device="cuda"), nb


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_split_fp32_out_with_beta(mdnn, dt, layout):
    for i, (m, n, k) in enumerate(SPLIT_SHAPES):
        sa, sb = _shapes(layout, m, n, k)
        a = W.normal(sa, 31, 10 * i + 1, dt, 1 / np.sqrt(k))
        b = W.normal(sb, 31, 10 * i + 2, dt)
        c = W.normal((m, n), 31, 10 * i + 3, "f32")
        ws, _ = _ws(mdnn, dt, m, n, k)
        got = _run(mdnn, layout, dev(a, dt), dev(b, dt), "f32", m, n, k, ws, beta=0.5, Cm=dev(c, "f32"))
        a64, b64 = decode(a, dt), decode(b, dt)
        want = ops.gemm(layout, a64, b64, 1.0, 0.5, c.astype(np.float64))
        assert norm_max_err(got, want) <= TOL, (m, n, k)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_split_lowp_out_bias_relu(mdnn, dt, layout):
    for i, (m, n, k) in enumerate(SPLIT_SHAPES):
        sa, sb = _shapes(layout, m, n, k)
        a = W.normal(sa, 32, 10 * i + 1, dt, 1 / np.sqrt(k))
        b = W.normal(sb, 32, 10 * i + 2, dt)
        bias = W.normal((n,), 32, 10 * i + 3, "f32", 0.5)
        ws, _ = _ws(mdnn, dt, m, n, k)
        got = _run(mdnn, layout, dev(a, dt), dev(b, dt), dt, m, n, k, ws, bias=dev(bias, "f32"), act=1)
        a64, b64 = decode(a, dt), decode(b, dt)
        exact = ops.bias_act(ops.gemm(layout, a64, b64), bias.astype(np.float64), "relu")
        err = accum_bound(ops.gemm(layout, np.abs(a64), np.abs(b64)) + np.abs(bias), k + 1)
        assert lowp_close(got, exact, dt, err), (m, n, k)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_split_relu_mask(mdnn, dt):
    """Backward-data form (NT) with the ReLU mask on the split path."""
    for i, (m, n, k) in enumerate([(256, 1024, 3136), (70, 136, 1000)]):
        dz = W.normal((m, k), 33, 10 * i + 1, dt, 1 / np.sqrt(k))
        w = W.normal((n, k), 33, 10 * i + 2, dt)
        y_in = W.normal((m, n), 33, 10 * i + 3, dt)
        ws, _ = _ws(mdnn, dt, m, n, k)
        got = _run(mdnn, "NT", dev(dz, dt), dev(w, dt), dt, m, n, k, ws, mask=dev(y_in, dt))
        dz64, w64 = decode(dz, dt), decode(w, dt)
        exact = np.where(decode(y_in, dt) > 0, ops.gemm("NT", dz64, w64), 0.0)
        err = accum_bound(np.abs(dz64) @ np.abs(w64).T, k)
        assert lowp_close(got, exact, dt, err)
        assert np.all(got[decode(y_in, dt) <= 0] == 0)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_split_integer_exact_and_deterministic(mdnn, dt):
    for layout in ("NN", "NT", "TN"):
        for i, (m, n, k) in enumerate(SPLIT_SHAPES):
            sa, sb = _shapes(layout, m, n, k)
            a = W.small_ints(sa, 34, 10 * i + 1, dtype=dt)
            b = W.small_ints(sb, 34, 10 * i + 2, dtype=dt)
            A, B = dev(a, dt), dev(b, dt)
            ws, _ = _ws(mdnn, dt, m, n, k)
            g1 = _run(mdnn, layout, A, B, "f32", m, n, k, ws)
            g2 = _run(mdnn, layout, A, B, "f32", m, n, k, ws)
            assert np.array_equal(g1, ops.gemm(layout, decode(a, dt), decode(b, dt))), (layout, m, n, k)
            assert np.array_equal(g1, g2)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_short_workspace_is_the_plain_gemm(mdnn, dt):
    """Too small a workspace, or none: bitwise the result of mdnn_gemm_mixed."""
    m, n, k = 256, 10, 1024
    a = W.normal((m, k), 35, 1, dt)
    b = W.normal((k, n), 35, 2, dt)
    A, B = dev(a, dt), dev(b, dt)
    plain = _run(mdnn, "NN", A, B, "f32", m, n, k, None)
    ws, nb = _ws(mdnn, dt, m, n, k, short=(1 << 40))   # 16 bytes: below any plan
    assert ws.numel() < nb
    assert np.array_equal(_run(mdnn, "NN", A, B, "f32", m, n, k, ws), plain)
    # a shape that plans no split (K < 256 for fp16 / bf16, 64 tiles for
    # fp32): the workspace is ignored
    m2, n2, k2 = 512, 512, 192
    a2 = W.normal((m2, k2), 35, 3, dt)
    b2 = W.normal((k2, n2), 35, 4, dt)
    A2, B2 = dev(a2, dt), dev(b2, dt)
    ws2, _ = _ws(mdnn, dt, 256, 1024, 3136)
    assert np.array_equal(_run(mdnn, "NN", A2, B2, "f32", m2, n2, k2, ws2),
                          _run(mdnn, "NN", A2, B2, "f32", m2, n2, k2, None))
