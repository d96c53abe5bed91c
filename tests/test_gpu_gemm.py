"""GPU parity of mdnn_gemm_mixed against the oracle (section 3.2, D = C + A*B).

fp32 outputs: normalized max error <= 1e-4 against the fp64 oracle on the same
input bits.  Low-precision outputs: within one storage ulp of the oracle's
rounding plus the fp32 accumulation bound gamma_K * sum |a||b| (the bound
matters where the result cancels to far below the operands' scale).  Small-integer operands: bit-exact.  Every tile configuration and
layout is exercised on ragged shapes; the full-size sweep (1024/4096/8192 in
NN/NT/TN, the launch configuration the benchmark times) is checked on sampled
rows and columns computed one by one by the oracle.
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


def _shapes(layout, m, n, k):
    a = (k, m) if layout == "TN" else (m, k)
    b = (n, k) if layout == "NT" else (k, n)
    return a, b


def _run(mdnn, layout, A, B, out_dt, m, n, k, bias=None, act=0, mask=None, alpha=1.0, beta=0.0,
         Cm=None, ld_pad=0):
    import torch
    D = empty((m, n + ld_pad), out_dt)
    D.fill_(float("nan"))
    mdnn.mdnn_gemm_mixed(LAYOUT[layout], m, n, k, alpha, A, A.stride(0), B, B.stride(0),
                         mdnn.dtype_of(A), beta, Cm, Cm.stride(0) if Cm is not None else 0, D,
                         D.stride(0), DT[out_dt], bias, act, mask,
                         mask.stride(0) if mask is not None else 0)
    torch.cuda.synchronize()
    return host64(D)[:, :n]


RAGGED = [(1, 1, 1), (7, 33, 100), (100, 7, 33), (33, 100, 7), (130, 70, 200), (300, 260, 129),
          (257, 513, 64), (64, 64, 1000)]


@pytest.mark.parametrize("tile", [1, 2, 3])
@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_gemm_ragged_all_tiles(mdnn, tile, dt, layout):
    mdnn.mdnn_set_gemm_tile(tile)
    try:
        for i, (m, n, k) in enumerate(RAGGED):
            sa, sb = _shapes(layout, m, n, k)
            a = W.normal(sa, 7, 10 * i + 1, dt, 1 / np.sqrt(k))
            b = W.normal(sb, 7, 10 * i + 2, dt, 1 / np.sqrt(k))
            got = _run(mdnn, layout, dev(a, dt), dev(b, dt), "f32", m, n, k)
            want = ops.gemm(layout, decode(a, dt), decode(b, dt))
            err = norm_max_err(got, want)
            assert err <= TOL, (tile, layout, dt, (m, n, k), err)
    finally:
        mdnn.mdnn_set_gemm_tile(0)


# shapes the direct-to-LDS pipelined kernel accepts (K % 64 == 0, M and N
# multiples of 8) but that are ragged with respect to its 256 x 256 and
# 128 x 128 tiles
PIPE = [(312, 264, 192), (520, 776, 320), (1000, 1032, 448), (8, 8, 64), (64, 2056, 128),
        (264, 8, 1024)]


@pytest.mark.parametrize("tile", [4, 5])
@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_gemm_pipelined_kernel_ragged(mdnn, dt, layout, tile):
    mdnn.mdnn_set_gemm_tile(tile)
    try:
        for i, (m, n, k) in enumerate(PIPE):
            sa, sb = _shapes(layout, m, n, k)
            a = W.normal(sa, 9, 10 * i + 1, dt, 1 / np.sqrt(k))
            b = W.normal(sb, 9, 10 * i + 2, dt, 1 / np.sqrt(k))
            got = _run(mdnn, layout, dev(a, dt), dev(b, dt), "f32", m, n, k)
            want = ops.gemm(layout, decode(a, dt), decode(b, dt))
            assert norm_max_err(got, want) <= TOL, (layout, dt, (m, n, k))
        # epilogues on the pipelined kernel: bias + ReLU to the storage type
        m, n, k = 520, 776, 320
        sa, sb = _shapes(layout, m, n, k)
        a = W.normal(sa, 9, 101, dt, 1 / np.sqrt(k))
        b = W.normal(sb, 9, 102, dt)
        bias = W.normal((n,), 9, 103, "f32", 0.5)
        got = _run(mdnn, layout, dev(a, dt), dev(b, dt), dt, m, n, k, bias=dev(bias, "f32"), act=1)
        a64, b64 = decode(a, dt), decode(b, dt)
        exact = ops.bias_act(ops.gemm(layout, a64, b64), bias.astype(np.float64), "relu")
        err = accum_bound(ops.gemm(layout, np.abs(a64), np.abs(b64)) + np.abs(bias), k + 1)
        assert lowp_close(got, exact, dt, err)
        # and the ReLU mask of a backward-data product
        y_in = W.normal((m, n), 9, 104, dt)
        got = _run(mdnn, layout, dev(a, dt), dev(b, dt), dt, m, n, k, mask=dev(y_in, dt))
        exact = np.where(decode(y_in, dt) > 0, ops.gemm(layout, a64, b64), 0.0)
        err = accum_bound(ops.gemm(layout, np.abs(a64), np.abs(b64)), k)
        assert lowp_close(got, exact, dt, err)
    finally:
        mdnn.mdnn_set_gemm_tile(0)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_gemm_pipelined_64x64_tiles(mdnn, dt, layout):
    """Grids of fewer than 128 tiles of 128 x 128 but at least 128 of 64 x 64
    (chosen automatically): ragged shapes, fp32 output, and the bias + ReLU
    and ReLU-mask epilogues stored in the storage type."""
    for i, (m, n, k) in enumerate([(1000, 1032, 448), (760, 1096, 192), (1024, 1024, 1024)]):
        sa, sb = _shapes(layout, m, n, k)
        a = W.normal(sa, 11, 10 * i + 1, dt, 1 / np.sqrt(k))
        b = W.normal(sb, 11, 10 * i + 2, dt, 1 / np.sqrt(k))
        got = _run(mdnn, layout, dev(a, dt), dev(b, dt), "f32", m, n, k)
        a64, b64 = decode(a, dt), decode(b, dt)
        want = ops.gemm(layout, a64, b64)
        assert norm_max_err(got, want) <= TOL, (layout, dt, (m, n, k))
        bias = W.normal((n,), 11, 10 * i + 3, "f32", 0.5)
        got = _run(mdnn, layout, dev(a, dt), dev(b, dt), dt, m, n, k, bias=dev(bias, "f32"), act=1)
        exact = ops.bias_act(want, bias.astype(np.float64), "relu")
        err = accum_bound(ops.gemm(layout, np.abs(a64), np.abs(b64)) + np.abs(bias), k + 1)
        assert lowp_close(got, exact, dt, err)
        y_in = W.normal((m, n), 11, 10 * i + 4, dt)
        got = _run(mdnn, layout, dev(a, dt), dev(b, dt), dt, m, n, k, mask=dev(y_in, dt))
        exact = np.where(decode(y_in, dt) > 0, want, 0.0)
        err = accum_bound(ops.gemm(layout, np.abs(a64), np.abs(b64)), k)
        assert lowp_close(got, exact, dt, err)


@pytest.mark.parametrize("tile", [1, 2, 4, 5])
@pytest.mark.parametrize("out_dt", ["f32", "f16"])
def test_gemm_every_epilogue_term_interior_and_edge_tiles(mdnn, tile, out_dt):
    """alpha, beta * C, bias, ReLU and the ReLU mask together, on a shape whose
    interior tiles take the straight-line store (4-aligned rows of D, C and
    the mask, aligned bias) and whose edge tiles take the bounded one, in the
    general (tile 1, 2) and pipelined (4, 5) kernels."""
    dt = "f16"
    m, n, k = 520, 776, 320
    mdnn.mdnn_set_gemm_tile(tile)
    try:
        a = W.normal((m, k), 12, 1, dt, 1 / np.sqrt(k))
        b = W.normal((k, n), 12, 2, dt)
        c = W.normal((m, n), 12, 3, out_dt)
        bias = W.normal((n,), 12, 4, "f32", 0.5)
        y_in = W.normal((m, n), 12, 5, dt)
        got = _run(mdnn, "NN", dev(a, dt), dev(b, dt), out_dt, m, n, k, bias=dev(bias, "f32"), act=1,
                   mask=dev(y_in, dt), alpha=0.75, beta=-0.5, Cm=dev(c, out_dt))
        a64, b64, c64 = decode(a, dt), decode(b, dt), decode(c, out_dt)
        pre = 0.75 * ops.gemm("NN", a64, b64) - 0.5 * c64
        exact = np.where(decode(y_in, dt) > 0, ops.bias_act(pre, bias.astype(np.float64), "relu"), 0.0)
        err = accum_bound(0.75 * (np.abs(a64) @ np.abs(b64)) + 0.5 * np.abs(c64) + np.abs(bias), k + 2)
        if out_dt == "f32":
            assert np.all(np.abs(got - exact) <= err + 2.0 ** -23 * np.abs(exact))
        else:
            assert lowp_close(got, exact, dt, err)
        assert np.all(got[decode(y_in, dt) <= 0] == 0)
    finally:
        mdnn.mdnn_set_gemm_tile(0)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_gemm_small_integers_bit_exact(mdnn, dt, layout):
    m, n, k = 200, 136, 1000
    sa, sb = _shapes(layout, m, n, k)
    a = W.small_ints(sa, 3, 1, dtype=dt)
    b = W.small_ints(sb, 3, 2, dtype=dt)
    got = _run(mdnn, layout, dev(a, dt), dev(b, dt), "f32", m, n, k)
    want = ops.gemm(layout, decode(a, dt), decode(b, dt))
    assert np.array_equal(got, want)


def test_fp32_accumulation_all_ones(mdnn):
    """Section 3.2: fp16 products accumulated in fp32.  4096 ones sum to exactly
    4096 (an fp16 accumulator would stall at 2048); with beta = 1 and C = 1
    the result is 4097."""
    import torch
    k = 4096
    a = torch.ones((1, k), dtype=torch.float16, device="cuda")
    b = torch.ones((k, 1), dtype=torch.float16, device="cuda")
    got = _run(mdnn, "NN", a, b, "f32", 1, 1, k)
    assert got[0, 0] == 4096.0
    c = torch.ones((1, 1), dtype=torch.float32, device="cuda")
    got = _run(mdnn, "NN", a, b, "f32", 1, 1, k, beta=1.0, Cm=c)
    assert got[0, 0] == 4097.0


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_gemm_alpha_beta_leading_dims(mdnn, dt):
    import torch
    m, n, k = 150, 90, 77
    a = W.normal((m, k + 5), 4, 1, dt)          # lda = k + 5 (not a multiple of 8)
    b = W.normal((n, k + 8), 4, 2, dt)          # NT, ldb = k + 8
    c = W.normal((m, n + 3), 4, 3, "f32")
    A, B, Cm = dev(a, dt), dev(b, dt), dev(c, "f32")
    Av, Bv, Cv = A[:, :k], B[:, :k], Cm[:, :n]
    got = _run(mdnn, "NT", Av, Bv, "f32", m, n, k, alpha=0.5, beta=-2.0, Cm=Cv, ld_pad=4)
    want = ops.gemm("NT", decode(a, dt)[:, :k], decode(b, dt)[:, :k], 0.5, -2.0, c[:, :n].astype(np.float64))
    assert norm_max_err(got, want) <= TOL
    del torch


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_gemm_bias_relu_lowp_out(mdnn, dt):
    m, n, k = 260, 200, 300
    a = W.normal((m, k), 5, 1, dt, 1 / np.sqrt(k))
    b = W.normal((k, n), 5, 2, dt)
    bias = W.normal((n,), 5, 3, "f32", 0.5)
    got = _run(mdnn, "NN", dev(a, dt), dev(b, dt), dt, m, n, k, bias=dev(bias, "f32"), act=1)
    a64, b64 = decode(a, dt), decode(b, dt)
    exact = ops.bias_act(ops.gemm("NN", a64, b64), bias.astype(np.float64), "relu")
    err = accum_bound(np.abs(a64) @ np.abs(b64) + np.abs(bias), k + 1)
    assert lowp_close(got, exact, dt, err)
    assert np.all(got >= 0)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_gemm_relu_mask_epilogue(mdnn, dt):
    """Backward-data form with the ReLU derivative of the layer input fused."""
    m, n, k = 129, 140, 96
    dz = W.normal((m, k), 6, 1, dt)
    w = W.normal((n, k), 6, 2, dt)
    y_in = W.normal((m, n), 6, 3, dt)          # the stored layer input (mask source)
    got = _run(mdnn, "NT", dev(dz, dt), dev(w, dt), dt, m, n, k, mask=dev(y_in, dt))
    dz64, w64 = decode(dz, dt), decode(w, dt)
    exact = np.where(decode(y_in, dt) > 0, ops.gemm("NT", dz64, w64), 0.0)
    err = accum_bound(np.abs(dz64) @ np.abs(w64).T, k)
    assert lowp_close(got, exact, dt, err)
    assert np.all(got[decode(y_in, dt) <= 0] == 0)


# (70, 130, 200): one K group per tile; the others leave fewer than 128
# workgroups over K >= 256, so four K groups share each tile (a ragged last
# group at K = 784 and 1001).
@pytest.mark.parametrize("mnk", [(70, 130, 200), (64, 128, 784), (33, 10, 1001)])
def test_gemm_fp32_path(mdnn, mnk):
    for layout in ("NN", "NT", "TN"):
        m, n, k = mnk
        sa, sb = _shapes(layout, m, n, k)
        a = W.normal(sa, 8, 1, "f32")
        b = W.normal(sb, 8, 2, "f32")
        bias = W.normal((n,), 8, 3, "f32")
        got = _run(mdnn, layout, dev(a, "f32"), dev(b, "f32"), "f32", m, n, k, bias=dev(bias, "f32"), act=1)
        a64, b64 = a.astype(np.float64), b.astype(np.float64)
        want = ops.bias_act(ops.gemm(layout, a64, b64), bias.astype(np.float64), "relu")
        # fp32 inputs: each product rounds too, gamma_{k+1} covers it
        err = accum_bound(ops.gemm(layout, np.abs(a64), np.abs(b64)) + np.abs(bias), k + 1)
        assert np.all(np.abs(got - want) <= err)
        # and the per-output parity metric of fp32 results
        assert norm_max_err(got, want) <= 1e-4, layout


def test_gemm_fp32_k_groups_integer_exact(mdnn):
    """Four K groups per tile summed in a fixed order: small integers stay
    exact, so the result is bit-identical to the exact product."""
    m, n, k = 64, 128, 784
    for layout in ("NN", "NT", "TN"):
        sa, sb = _shapes(layout, m, n, k)
        a = W.small_ints(sa, 10, 1, dtype="f32")
        b = W.small_ints(sb, 10, 2, dtype="f32")
        got = _run(mdnn, layout, dev(a, "f32"), dev(b, "f32"), "f32", m, n, k)
        assert np.array_equal(got, ops.gemm(layout, a.astype(np.float64), b.astype(np.float64)))


def test_gemm_k_zero_and_empty(mdnn):
    import torch
    c = torch.full((3, 4), 2.0, dtype=torch.float32, device="cuda")
    a = torch.empty((3, 0), dtype=torch.float16, device="cuda")
    b = torch.empty((0, 4), dtype=torch.float16, device="cuda")
    got = _run(mdnn, "NN", a, b, "f32", 3, 4, 0, beta=0.5, Cm=c)
    assert np.all(got == 1.0)
    d = torch.empty((0, 4), dtype=torch.float32, device="cuda")
    mdnn.mdnn_gemm_mixed(0, 0, 4, 8, 1.0, None, 8, None, 4, 1, 0.0, None, 0, d, 4, 0)


@pytest.mark.parametrize("size", W.GEMM_SIZES)
@pytest.mark.parametrize("layout", W.GEMM_LAYOUTS)
def test_gemm_sweep_full_size_sampled(mdnn, size, layout):
    """The fp16 GEMM sweep at its full sizes, fp32 output, in the automatic
    tile configuration: 48 sampled rows and 48 sampled columns against the
    oracle, computed row by row / column by column."""
    import torch
    m = n = k = size
    a, b = W.gemm_operands(layout, m, n, k)
    A, B = dev(a, "f16"), dev(b, "f16")
    D = torch.empty((m, n), dtype=torch.float32, device="cuda")
    mdnn.mdnn_gemm_mixed(LAYOUT[layout], m, n, k, 1.0, A, A.stride(0), B, B.stride(0), 1, 0.0, None,
                         0, D, n, 0)
    torch.cuda.synchronize()
    rs = np.random.default_rng(size)
    rows = np.sort(rs.choice(m, 48, replace=False))
    cols = np.sort(rs.choice(n, 48, replace=False))
    a64, b64 = a.astype(np.float64), b.astype(np.float64)
    op_a = a64.T if layout == "TN" else a64
    op_b = b64.T if layout == "NT" else b64
    want_rows = op_a[rows] @ op_b
    want_cols = op_a @ op_b[:, cols]
    got = D.cpu().numpy().astype(np.float64)
    assert norm_max_err(got[rows], want_rows) <= TOL
    assert norm_max_err(got[:, cols], want_cols) <= TOL
    assert np.all(np.isfinite(got))


# Narrow shapes on the pipelined kernel (automatic choice): N <= 64 takes the
# 256 x 64 tile, M <= 64 the 64 x 256 tile, N <= 128 the 128 x 128 tile
# (a 256 x 256 tile would be mostly padding); ragged M / N included.
NARROW = [(8192, 64, 576), (4000, 48, 256), (64, 8192, 512), (40, 4096, 256), (16384, 128, 320)]


@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_gemm_narrow_shapes_pipelined(mdnn, layout):
    for i, (m, n, k) in enumerate(NARROW):
        sa, sb = _shapes(layout, m, n, k)
        a = W.normal(sa, 36, 10 * i + 1, "f16", 1 / np.sqrt(k))
        b = W.normal(sb, 36, 10 * i + 2, "f16")
        got = _run(mdnn, layout, dev(a, "f16"), dev(b, "f16"), "f32", m, n, k)
        want = ops.gemm(layout, decode(a, "f16"), decode(b, "f16"))
        assert norm_max_err(got, want) <= TOL, (layout, m, n, k)
        ai = W.small_ints(sa, 37, 10 * i + 1, dtype="bf16")
        bi = W.small_ints(sb, 37, 10 * i + 2, dtype="bf16")
        got = _run(mdnn, layout, dev(ai, "bf16"), dev(bi, "bf16"), "f32", m, n, k)
        assert np.array_equal(got, ops.gemm(layout, decode(ai, "bf16"), decode(bi, "bf16"))), (layout, m, n, k)
