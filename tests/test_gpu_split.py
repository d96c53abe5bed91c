"""GPU parity of the Eq. (1) split and the three-product fp32 GEMM (section 3.2).

The split is integer-like work (two RNE roundings of exact fp32 values): the
GPU's fp16 bits must equal the oracle's exactly.  The GEMM is compared with
the oracle's exact value of the three products (fp32 accumulation bound over
the 2K + 2 terms each output sums), with the exact fp64 product of the fp32
inputs (that bound plus 2^-20 of sum |a||b|, the split's own error), and with
a plain fp16 product of the same inputs, which it must beat by a wide margin.
"""
import numpy as np
import pytest

import workloads as W
from oracle import ops
from tests.helpers import accum_bound, dev, host64, norm_max_err

pytestmark = pytest.mark.gpu


def _fp32(shape, seed, tid, lo_exp=-6, hi_exp=6):
    g = W.rng(seed, tid)
    mant = g.uniform(1.0, 2.0, shape)
    e = g.integers(lo_exp, hi_exp, shape)
    sign = np.where(g.random(shape) < 0.5, -1.0, 1.0)
    return (sign * np.ldexp(mant, e)).astype(np.float32)


@pytest.mark.parametrize("rows, cols, scale", [(1, 1, 1.0), (37, 129, 1.0), (300, 260, 2.0 ** -3),
                                               (8, 1000, 2.0 ** 10), (513, 72, 0.5)])
def test_split_bit_exact(mdnn, rows, cols, scale):
    import torch
    x = _fp32((rows, cols + 5), 21, 1) * np.float32(scale)
    X = dev(x, "f32")[:, :cols]                          # leading dimension cols + 5
    hi, lo = mdnn.split_f16(X, scale)
    torch.cuda.synchronize()
    h, l = ops.split_f16(x[:, :cols].astype(np.float64), scale)
    assert np.array_equal(host64(hi), h)
    assert np.array_equal(host64(lo), l)


def test_split_fp16_inputs_have_zero_second_term(mdnn):
    import torch
    x = W.normal((64, 64), 22, 1, "f16").astype(np.float32)
    hi, lo = mdnn.split_f16(dev(x, "f32"), 1.0)
    torch.cuda.synchronize()
    assert np.array_equal(host64(hi), x.astype(np.float64)) and not host64(lo).any()


def _operands(layout, m, n, k, seed):
    sa = (k, m) if layout == "TN" else (m, k)
    sb = (n, k) if layout == "NT" else (k, n)
    return _fp32(sa, seed, 1), _fp32(sb, seed, 2)


SHAPES = [(300, 260, 520), (64, 64, 64), (1000, 1032, 448), (129, 77, 100), (8, 8, 8), (512, 512, 1024)]


@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_gemm_split3_against_oracle(mdnn, layout):
    import torch
    L = {"NN": mdnn.NN, "NT": mdnn.NT, "TN": mdnn.TN}[layout]
    for i, (m, n, k) in enumerate(SHAPES):
        a, b = _operands(layout, m, n, k, 30 + i)
        got = mdnn.gemm_split3(L, dev(a, "f32"), dev(b, "f32"))
        torch.cuda.synchronize()
        got = host64(got)
        a64, b64 = a.astype(np.float64), b.astype(np.float64)
        absprod = ops.gemm(layout, np.abs(a64), np.abs(b64))
        method = ops.gemm_split3(layout, a64, b64, 1.0, 1.0)
        assert np.all(np.abs(got - method) <= accum_bound(absprod, 2 * k + 2)), (layout, (m, n, k))
        exact = ops.gemm(layout, a64, b64)
        assert np.all(np.abs(got - exact) <= accum_bound(absprod, 2 * k + 2) + 2.0 ** -20 * absprod)
        # a plain fp16 product of the same data is far less accurate
        a16 = a.astype(np.float16).astype(np.float64)
        b16 = b.astype(np.float16).astype(np.float64)
        err16 = np.max(np.abs(ops.gemm(layout, a16, b16) - exact))
        assert np.max(np.abs(got - exact)) * 64 < err16


@pytest.mark.parametrize("case", ["large", "small", "subnormal", "zeros", "inf", "nan", "ragged"])
def test_split_scale_chosen_on_device(mdnn, case):
    """scale 0: the library picks the power of two from max|x| on the device
    and writes it out; the split is then bit-exact at that scale."""
    import torch
    rows, cols = (37, 129) if case == "ragged" else (64, 200)
    x = {"large": lambda: _fp32((rows, cols), 23, 1, 18, 22),
         "small": lambda: _fp32((rows, cols), 23, 2, -30, -26),
         "subnormal": lambda: _fp32((rows, cols), 23, 3, -140, -130),
         "zeros": lambda: np.zeros((rows, cols), np.float32),
         "inf": lambda: _fp32((rows, cols), 23, 4),
         "nan": lambda: _fp32((rows, cols), 23, 5),
         "ragged": lambda: _fp32((rows, cols), 23, 6, -3, 9)}[case]()
    if case == "inf":
        x[5, 7] = np.inf
    if case == "nan":
        x[rows - 1, cols - 1] = np.nan
    want = ops.split_scale(x)
    assert {"large": 2.0 ** 7, "small": 2.0 ** -41, "zeros": 1.0, "inf": 1.0, "nan": 1.0,
            "subnormal": 2.0 ** -126}.get(case, want) == want
    hi, lo, s = mdnn.split_f16(dev(x, "f32"), 0.0)
    torch.cuda.synchronize()
    assert float(s.item()) == want
    h, l = ops.split_f16(x.astype(np.float64), want)
    fin = np.isfinite(x)
    assert np.array_equal(host64(hi)[fin], h[fin]) and np.array_equal(host64(lo)[fin], l[fin])


@pytest.mark.parametrize("auto", [False, True])
def test_gemm_split3_alpha_beta_scales_and_aliasing(mdnn, auto):
    """alpha / beta with C aliasing D, power-of-two scales that bring data of
    large and small magnitude into fp16's range (given, or chosen on the
    device), and K = 0."""
    import torch
    m, n, k = 200, 136, 320
    a = _fp32((m, k), 40, 1, 18, 22)                    # |a| ~ 2^18 .. 2^22: beyond fp16
    b = _fp32((k, n), 40, 2, -30, -26)                  # |b| ~ 2^-30: below fp16's normals
    c = _fp32((m, n), 40, 3)
    A, B = dev(a, "f32"), dev(b, "f32")
    sa, sb = ops.split_scale(a), ops.split_scale(b)
    assert sa == 2.0 ** 7 and sb == 2.0 ** -41
    D = dev(c, "f32")
    if auto:
        mdnn.gemm_split3(mdnn.NN, A, B, 0.0, 0.0, alpha=0.75, beta=-1.5, Cm=D, out=D)
    else:
        mdnn.gemm_split3(mdnn.NN, A, B, sa, sb, alpha=0.75, beta=-1.5, Cm=D, out=D)
    torch.cuda.synchronize()
    a64, b64, c64 = a.astype(np.float64), b.astype(np.float64), c.astype(np.float64)
    absprod = ops.gemm("NN", np.abs(a64), np.abs(b64))
    method = ops.gemm_split3("NN", a64, b64, sa, sb, 0.75, -1.5, c64)
    bound = accum_bound(0.75 * absprod + 1.5 * np.abs(c64), 2 * k + 3)
    assert np.all(np.abs(host64(D) - method) <= bound)
    # K = 0: D = beta C
    E = dev(c, "f32")
    out = torch.empty((m, n), dtype=torch.float32, device="cuda")
    mdnn.gemm_split3(mdnn.NN, A[:, :0], B[:0, :], beta=2.0, Cm=E, out=out)
    torch.cuda.synchronize()
    assert np.array_equal(host64(out), 2.0 * c64)


def test_gemm_split3_full_size_sampled(mdnn):
    """4096^3 NN as the benchmark runs it: 48 sampled rows against fp64."""
    import torch
    m = n = k = 4096
    a, b = _operands("NN", m, n, k, 50)
    got = mdnn.gemm_split3(mdnn.NN, dev(a, "f32"), dev(b, "f32"))
    torch.cuda.synchronize()
    rows = W.rng(50, 9).choice(m, 48, replace=False)
    a64, b64 = a[rows].astype(np.float64), b.astype(np.float64)
    exact = a64 @ b64
    absprod = np.abs(a64) @ np.abs(b64)
    sel = host64(got)[rows]
    assert np.all(np.abs(sel - exact) <= accum_bound(absprod, 2 * k + 2) + 2.0 ** -20 * absprod)
    assert norm_max_err(sel, exact) < 1e-6
