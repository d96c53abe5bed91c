"""GPU parity of the skinny products (section 3.2's D = C + A*B with one tiny
dimension): N <= 4 with A K-contiguous (a regression head), TN with N <= 16
(the weight gradient of a narrow head, K split over a workspace or not), and
K <= 4 in every layout (back-propagation through a regression head).  The
other shapes listed (N = 10 or 16, K = 10 or 16) sit next to those limits and
run on the general kernels.

Same bars as the other GEMM tests: fp32 outputs within 1e-4 normalized max
error of the fp64 oracle, low-precision outputs within one storage ulp plus
gamma_K * sum |a||b|, small integers bit-exact, repeated calls bitwise equal.
Shapes include the workloads' heads (4096 x 1 x 4096, 256 x 10 x 1024,
64 x 10 x 128, 4096 x 4096 x 1) plus ragged M, N = 1..16, K = 1..4 and K not
a multiple of 8, and leading dimensions wider than the rows.
"""
import numpy as np
import pytest

import workloads as W
from oracle import ops
from oracle.rounding import decode, round_to
from tests.helpers import DT, accum_bound, dev, empty, host64, lowp_close, norm_max_err, ulp

pytestmark = pytest.mark.gpu

LAYOUT = {"NN": 0, "NT": 1, "TN": 2}
TOL = 1e-4
SHAPES = {  # layout -> (m, n, k) list
    "NN": [(4096, 1, 4096), (1001, 1, 1000), (256, 10, 1024), (64, 10, 128), (77, 16, 301), (5, 3, 40), (300, 2, 17),
           (129, 4, 700), (333, 50, 3)],
    "NT": [(256, 10, 1024), (130, 1, 4600), (131, 3, 500), (9, 1, 23), (1000, 4096, 1), (70, 33, 10), (64, 128, 4)],
    "TN": [(4096, 1, 4096), (1536, 1, 1000), (1024, 10, 256), (128, 10, 64), (1001, 3, 300), (37, 16, 1000), (9, 5, 20),
           (700, 9, 16), (500, 64, 2)],
}
CASES = [(lay, s) for lay, lst in SHAPES.items() for s in lst]


def _shapes(layout, m, n, k):
    return ((k, m) if layout == "TN" else (m, k)), ((n, k) if layout == "NT" else (k, n))


def _run(mdnn, layout, A, B, out_dt, m, n, k, ws=None, bias=None, act=0, mask=None, beta=0.0, Cm=None, ld_pad=0):
    import torch
    D = empty((m, n + ld_pad), out_dt)
    D.fill_(float("nan"))
    args = (LAYOUT[layout], m, n, k, 1.0, A, A.stride(0), B, B.stride(0), mdnn.dtype_of(A), beta, Cm,
            Cm.stride(0) if Cm is not None else 0, D, D.stride(0), DT[out_dt], bias, act, mask,
            mask.stride(0) if mask is not None else 0)
    if ws is None:
        mdnn.mdnn_gemm_mixed(*args)
    else:
        mdnn.mdnn_gemm_mixed_ws(*args, ws, ws.numel())
    torch.cuda.synchronize()
    return host64(D)[:, :n]


def _ws(mdnn, dt, m, n, k):
    import torch
    nb = mdnn.mdnn_gemm_workspace(DT[dt], m, n, k)
    return torch.empty((max(nb, 16),), dtype=torch.uint8, device="cuda")


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("case", CASES, ids=[f"{l}-{m}x{n}x{k}" for l, (m, n, k) in CASES])
def test_skinny_fp32_out_beta(mdnn, dt, case):
    layout, (m, n, k) = case
    sa, sb = _shapes(layout, m, n, k)
    a = W.normal(sa, 41, 1, dt, 1 / np.sqrt(k))
    b = W.normal(sb, 41, 2, dt)
    c = W.normal((m, n), 41, 3, "f32")
    A, B, Cm = dev(a, dt), dev(b, dt), dev(c, "f32")
    a64, b64 = decode(a, dt), decode(b, dt)
    want = ops.gemm(layout, a64, b64, 1.0, -0.5, c.astype(np.float64))
    for ws in (None, _ws(mdnn, dt, m, n, k)):
        got = _run(mdnn, layout, A, B, "f32", m, n, k, ws=ws, beta=-0.5, Cm=Cm)
        assert norm_max_err(got, want) <= TOL, (layout, m, n, k, ws is None)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_skinny_lowp_bias_relu_and_mask(mdnn, dt, layout):
    for i, (m, n, k) in enumerate(SHAPES[layout]):
        sa, sb = _shapes(layout, m, n, k)
        a = W.normal(sa, 42, 10 * i + 1, dt, 1 / np.sqrt(k))
        b = W.normal(sb, 42, 10 * i + 2, dt)
        bias = W.normal((n,), 42, 10 * i + 3, "f32", 0.5)
        y_in = W.normal((m, n), 42, 10 * i + 4, dt)
        a64, b64 = decode(a, dt), decode(b, dt)
        got = _run(mdnn, layout, dev(a, dt), dev(b, dt), dt, m, n, k, ws=_ws(mdnn, dt, m, n, k),
                   bias=dev(bias, "f32"), act=1)
        exact = ops.bias_act(ops.gemm(layout, a64, b64), bias.astype(np.float64), "relu")
        err = accum_bound(ops.gemm(layout, np.abs(a64), np.abs(b64)) + np.abs(bias), k + 1)
        assert lowp_close(got, exact, dt, err), (layout, m, n, k)
        got = _run(mdnn, layout, dev(a, dt), dev(b, dt), dt, m, n, k, mask=dev(y_in, dt), ld_pad=3)
        exact = np.where(decode(y_in, dt) > 0, ops.gemm(layout, a64, b64), 0.0)
        err = accum_bound(ops.gemm(layout, np.abs(a64), np.abs(b64)), k)
        assert lowp_close(got, exact, dt, err), (layout, m, n, k)
        assert np.all(got[decode(y_in, dt) <= 0] == 0)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_skinny_integer_exact_and_deterministic(mdnn, dt):
    for layout, lst in SHAPES.items():
        for i, (m, n, k) in enumerate(lst):
            sa, sb = _shapes(layout, m, n, k)
            a = W.small_ints(sa, 43, 10 * i + 1, dtype=dt)
            b = W.small_ints(sb, 43, 10 * i + 2, dtype=dt)
            A, B = dev(a, dt), dev(b, dt)
            ws = _ws(mdnn, dt, m, n, k)
            g1 = _run(mdnn, layout, A, B, "f32", m, n, k, ws=ws)
            g2 = _run(mdnn, layout, A, B, "f32", m, n, k, ws=ws)
            assert np.array_equal(g1, ops.gemm(layout, decode(a, dt), decode(b, dt))), (layout, m, n, k)
            assert np.array_equal(g1, g2)


def test_skinny_strided_operands(mdnn):
    """Leading dimensions wider than the rows and an unaligned A view (the
    element-wise load paths)."""
    import torch
    m, n, k = 203, 3, 333
    a = W.normal((m, k + 9), 44, 1, "f16")
    b = W.normal((k, n + 6), 44, 2, "f16")
    A, B = dev(a, "f16")[:, 1:k + 1], dev(b, "f16")[:, :n]
    got = _run(mdnn, "NN", A, B, "f32", m, n, k)
    want = ops.gemm("NN", decode(a, "f16")[:, 1:k + 1], decode(b, "f16")[:, :n])
    assert norm_max_err(got, want) <= TOL
    n = 10
    at = W.normal((k, m + 5), 44, 3, "bf16")
    bt = W.normal((k, n + 2), 44, 4, "bf16")
    At, Bt = dev(at, "bf16")[:, 1:m + 1], dev(bt, "bf16")[:, :n]
    got = _run(mdnn, "TN", At, Bt, "f32", m, n, k, ws=_ws(mdnn, "bf16", m, n, k))
    want = ops.gemm("TN", decode(at, "bf16")[:, 1:m + 1], decode(bt, "bf16")[:, :n])
    assert norm_max_err(got, want) <= TOL
    del torch


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
@pytest.mark.parametrize("mnk", [(1001, 4096, 1), (4096, 4100, 3), (37, 64, 2)], ids=["ragged_m", "ragged_n", "small"])
def test_skinny_depth_relu_mask_rows_in_flight(mdnn, dt, layout, mnk):
    """The outer-product kernel (K <= 4) with only a ReLU mask after the
    product and contiguous 8-aligned rows: four rows' mask runs loaded ahead
    of their stores (rows beyond M, and columns past the last whole run of
    eight, on the row-at-a-time path).  Masked entries are 0 even where the
    incoming gradient is Inf."""
    m, n, k = mnk
    sa, sb = _shapes(layout, m, n, k)
    a = W.normal(sa, 43, 1, dt, 1.0)
    b = W.normal(sb, 43, 2, dt)
    y_in = W.normal((m, n), 43, 3, dt)
    a64, b64 = decode(a, dt), decode(b, dt)
    # an Inf in A: its products are masked to 0 wherever y_in <= 0
    ai = np.array(a, copy=True)
    inf = 0x7F80 if dt == "bf16" else np.inf  # bf16 is stored as bit patterns
    if layout == "TN":
        ai[0, 5] = inf
    else:
        ai[5, 0] = inf
    a64i = decode(ai, dt)
    got = _run(mdnn, layout, dev(ai, dt), dev(b, dt), dt, m, n, k, mask=dev(y_in, dt))
    # the same product with a padded output row (the row-at-a-time path): the same bits
    slow = _run(mdnn, layout, dev(ai, dt), dev(b, dt), dt, m, n, k, mask=dev(y_in, dt), ld_pad=3)
    same = (got == slow) | (np.isnan(got) & np.isnan(slow))
    assert np.all(same), [(i, got.flat[i], slow.flat[i]) for i in np.flatnonzero(~same)[:5]]
    keep = decode(y_in, dt) > 0
    with np.errstate(invalid="ignore"):
        prod = ops.gemm(layout, a64i, b64)
    exact = np.where(keep, prod, 0.0)
    assert np.all(got[~keep] == 0)
    fin = np.isfinite(exact)
    err = accum_bound(ops.gemm(layout, np.abs(a64), np.abs(b64)), k)
    if dt == "f32":
        assert np.all(np.abs(got[fin] - exact[fin]) <= err[fin] + 1e-30)
    else:
        ok = np.abs(got[fin] - round_to(exact[fin], dt)) <= ulp(np.abs(exact[fin]), dt) + err[fin]
        bad = np.flatnonzero(~ok)[:5]
        assert lowp_close(got[fin], exact[fin], dt, err[fin]), [(got[fin][i], exact[fin][i]) for i in bad]
    assert np.all(~np.isfinite(got[~fin])) and np.all(np.sign(got[~fin]) == np.sign(exact[~fin]))
