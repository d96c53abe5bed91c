"""Pins of the oracle's Eq. (1) split (section 3.2, reduced and mixed precision).

The split of an fp32 value x at scale s is x ~ s*X1 + s*2^-11*X2 with X1 and X2
fp16 numbers.  Pins: the paper's constant (s2 = 2^-11 s1), hand-derived splits
(ties to even included), exactness for fp16-representable inputs, the
reconstruction error bound (22 significant bits), power-of-two scale and sign
invariance, and the three-product GEMM against the exact four-product
identity and the exact fp64 product.
"""
import numpy as np
import pytest

from oracle import ops

F16_MAX = 65504.0


def test_paper_constant():
    # section 3.2: a well-scaled matrix splits with a2 = 2^-11 * a1
    assert ops.SPLIT_SHIFT == 2.0 ** -11


@pytest.mark.parametrize("x, hi, lo", [
    (3.0, 3.0, 0.0),                                  # fp16 number: no second term
    (1.0 + 2.0 ** -11, 1.0, 1.0),                     # tie: X1 rounds to even (1), X2 = 1
    (1.0 + 3 * 2.0 ** -11, 1.0 + 2.0 ** -9, -1.0),    # tie up to the even neighbour, X2 = -1
    (-(1.0 + 2.0 ** -11), -1.0, -1.0),
    # fp32(1/3) = 11184811 * 2^-25: X1 = 1365 * 2^-12; remainder 2731 * 2^-25,
    # times 2^11 = 1365.5 * 2^-13, a tie that rounds to 1366 * 2^-13
    (11184811 * 2.0 ** -25, 1365 * 2.0 ** -12, 1366 * 2.0 ** -13),
])
def test_hand_derived_splits(x, hi, lo):
    h, l = ops.split_f16(np.array([x]), 1.0)
    assert h[0] == hi and l[0] == lo


def _fp32(g, shape, lo_exp, hi_exp):
    mant = g.uniform(1.0, 2.0, shape)
    e = g.integers(lo_exp, hi_exp, shape)
    sign = np.where(g.random(shape) < 0.5, -1.0, 1.0)
    return (sign * np.ldexp(mant, e)).astype(np.float32).astype(np.float64)


def test_reconstruction_keeps_22_bits():
    g = np.random.default_rng(5)
    x = _fp32(g, 20000, -10, 14)
    hi, lo = ops.split_f16(x, 1.0)
    rec = hi + ops.SPLIT_SHIFT * lo
    assert np.all(np.abs(x - rec) <= 2.0 ** -22 * np.abs(x))
    # X1 alone keeps 11 bits, so the second term carries real information
    assert np.max(np.abs(x - hi) / np.abs(x)) > 2.0 ** -13


def test_fp16_values_have_no_second_term():
    g = np.random.default_rng(6)
    x = g.standard_normal(5000).astype(np.float16).astype(np.float64)
    hi, lo = ops.split_f16(x, 1.0)
    assert np.array_equal(hi, x) and np.all(lo == 0.0)


@pytest.mark.parametrize("k", [-20, -3, 5, 30])
def test_power_of_two_scale_and_sign(k):
    g = np.random.default_rng(7)
    x = _fp32(g, 4000, -8, 12)
    h1, l1 = ops.split_f16(x * 2.0 ** k, 2.0 ** k)
    h0, l0 = ops.split_f16(x, 1.0)
    assert np.array_equal(h1, h0) and np.array_equal(l1, l0)
    hn, ln = ops.split_f16(-x, 1.0)
    assert np.array_equal(hn, -h0) and np.array_equal(ln, -l0)


@pytest.mark.parametrize("mx, want", [
    (1.0, 2.0 ** -14),                 # 1 / 2^-14 = 2^14: the bottom of [2^14, 2^15)
    (1.9990234375, 2.0 ** -14),        # just below 2: still exponent 0
    (2.0, 2.0 ** -13),
    (65504.0, 2.0),                    # fp16's largest finite value -> 32752
    (65536.0, 4.0),
    (-3.0, 2.0 ** -13),                # the magnitude decides
    (1.5 * 2.0 ** -130, 2.0 ** -126),  # the floor: an fp32 subnormal maximum
    (2.0 ** -112, 2.0 ** -126),        # exponent -126 exactly
    (2.0 ** -111, 2.0 ** -125),
    (0.0, 1.0), (np.inf, 1.0), (-np.inf, 1.0), (np.nan, 1.0),
])
def test_split_scale_rule(mx, want):
    """The scale chosen for Eq. (1) when the caller leaves it open, on
    hand-picked maxima (the other entries are smaller)."""
    x = np.array([0.25 * abs(mx) if np.isfinite(mx) else 0.0, mx, 0.0])
    assert ops.split_scale(x) == want


def test_split_scale_puts_the_maximum_in_range():
    """Property of the chosen scale on random data of any magnitude: the
    largest |X| / s lies in [2^14, 2^15), a power of two, exact."""
    g = np.random.default_rng(11)
    for lo_e, hi_e in ((-100, -90), (-20, -5), (-1, 1), (10, 20), (100, 120)):
        x = _fp32(g, 500, lo_e, hi_e)
        s = ops.split_scale(x)
        assert np.frexp(s)[0] == 0.5
        r = np.max(np.abs(x)) / s
        assert 2.0 ** 14 <= r < 2.0 ** 15


def test_scale_brings_large_values_into_fp16_range():
    g = np.random.default_rng(8)
    x = _fp32(g, 1000, 20, 30)                     # far beyond fp16's range
    s = ops.split_scale(x)
    hi, lo = ops.split_f16(x, s)
    assert np.max(np.abs(hi)) < F16_MAX
    rec = s * (hi + ops.SPLIT_SHIFT * lo)
    assert np.all(np.abs(x - rec) <= 2.0 ** -22 * np.abs(x))


@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_three_products_against_four_and_exact(layout):
    g = np.random.default_rng(9)
    m, n, k = 17, 13, 40
    a = g.standard_normal((k, m) if layout == "TN" else (m, k)).astype(np.float32).astype(np.float64)
    b = g.standard_normal((n, k) if layout == "NT" else (k, n)).astype(np.float32).astype(np.float64)
    sa, sb = 2.0 ** -2, 2.0 ** 3
    d3 = ops.gemm_split3(layout, a, b, sa, sb)
    a1, a2 = ops.split_f16(a, sa)
    b1, b2 = ops.split_f16(b, sb)
    ra = sa * a1 + sa * ops.SPLIT_SHIFT * a2
    rb = sb * b1 + sb * ops.SPLIT_SHIFT * b2
    # adding back the dropped X2*Y2 product gives the product of the two
    # reconstructions (up to fp64 rounding)
    d4 = d3 + (sa * sb * ops.SPLIT_SHIFT ** 2) * ops.gemm(layout, a2, b2)
    full = ops.gemm(layout, ra, rb)
    assert np.max(np.abs(d4 - full)) <= 1e-13 * np.max(np.abs(full))
    # and the three products stay within 2^-20 of the exact product
    bound = ops.gemm(layout, np.abs(a), np.abs(b))
    assert np.all(np.abs(d3 - ops.gemm(layout, a, b)) <= 2.0 ** -20 * bound)


def test_alpha_beta():
    g = np.random.default_rng(10)
    a = g.standard_normal((6, 5)).astype(np.float32).astype(np.float64)
    b = g.standard_normal((5, 4)).astype(np.float32).astype(np.float64)
    c = g.standard_normal((6, 4))
    d = ops.gemm_split3("NN", a, b, 1.0, 1.0, alpha=0.5, beta=-2.0, c=c)
    assert np.allclose(d, 0.5 * ops.gemm_split3("NN", a, b, 1.0, 1.0) - 2.0 * c, rtol=0, atol=1e-14)
    # beta == 0 never reads C
    d0 = ops.gemm_split3("NN", a, b, 1.0, 1.0, beta=0.0, c=np.full((6, 4), np.nan))
    assert np.all(np.isfinite(d0))
