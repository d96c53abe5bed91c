"""Pins of the Winograd F(2x2, 3x3) restatement (oracle/winograd.py).

* The 1-D algorithm F(2, 3): A^T [(G g) (.) (B^T d)] equals the two outputs
  of the 3-tap correlation of d with g, computed by hand -- a wrong entry in
  any of the three transform matrices breaks it.
* The 2-D algorithm reproduces the plain convolution (ops.conv2d_fwd) to
  fp64 rounding for same / valid padding, ragged last tiles (odd output
  sizes), one channel and several, and bit for bit on small integers.
* error_scale bounds the result (|sum| <= sum of |terms|), and a numpy
  emulation of a low-precision implementation (transforms rounded to fp16,
  products summed in fp32) stays within the bound the GPU test uses.
"""
import numpy as np
import pytest

from oracle import ops, winograd as wg
from oracle.rounding import round_to


def test_one_dimensional_f23():
    g = np.random.default_rng(1).standard_normal((50, 3))
    d = np.random.default_rng(2).standard_normal((50, 4))
    for gi, di in zip(g, d):
        y = wg.AT @ ((wg.G @ gi) * (wg.BT @ di))
        want = [di[0] * gi[0] + di[1] * gi[1] + di[2] * gi[2], di[1] * gi[0] + di[2] * gi[1] + di[3] * gi[2]]
        assert np.allclose(y, want, rtol=0, atol=1e-14)


@pytest.mark.parametrize("shape", [(2, 6, 6, 3, 4, 1), (1, 7, 5, 2, 3, 1), (2, 5, 8, 3, 2, 0), (1, 4, 4, 1, 1, 2),
                                   (3, 9, 9, 5, 6, 1), (1, 3, 3, 2, 2, 0)])
def test_matches_the_convolution(shape):
    n, h, w, c, k, pad = shape
    rng = np.random.default_rng(sum(shape))
    x = rng.standard_normal((n, h, w, c))
    f = rng.standard_normal((k, 3, 3, c))
    want = ops.conv2d_fwd(x, f, pad)
    got = wg.conv2d_fwd_winograd(x, f, pad)
    assert got.shape == want.shape
    assert np.max(np.abs(got - want)) <= 1e-12 * np.max(np.abs(want))


def test_small_integers_exact():
    rng = np.random.default_rng(7)
    x = rng.integers(-4, 5, (2, 8, 7, 3)).astype(np.float64)
    f = rng.integers(-4, 5, (5, 3, 3, 3)).astype(np.float64)
    assert np.array_equal(wg.conv2d_fwd_winograd(x, f, 1), ops.conv2d_fwd(x, f, 1))


def test_tiles_cover_the_output():
    for h, w, pad in [(6, 6, 1), (7, 5, 1), (3, 3, 0), (1, 1, 1), (8, 9, 2)]:
        ho, wo, th, tw = wg.tiles_hw(h, w, pad)
        assert (ho, wo) == ops.conv_out_hw(h, w, 3, 3, pad)
        assert 2 * th >= ho > 2 * th - 2 and 2 * tw >= wo > 2 * tw - 2


@pytest.mark.parametrize("fmt, c", [("f16", 64), ("bf16", 16)])
def test_low_precision_emulation_within_bound(fmt, c):
    """Transforms computed exactly then rounded to the storage format once
    (as the GPU kernels store them), the 16 products summed in fp32, the
    output transform in fp32: the error stays below
    (2u + u^2 + gamma_C (1 + u)^2 + gamma_9) * error_scale."""
    rng = np.random.default_rng(11)
    n, h, w, k, pad = 2, 10, 9, 8, 1
    x = round_to(rng.standard_normal((n, h, w, c)), fmt)
    f = round_to(rng.standard_normal((k, 3, 3, c)) / np.sqrt(9 * c), fmt)
    u = round_to(wg.filter_transform(f), fmt)
    v = round_to(wg.input_transform(wg.input_tiles(x, pad)), fmt)
    m = np.zeros(v.shape[:5] + (k,), dtype=np.float32)
    for ci in range(c):  # fp32 accumulation in channel order
        m = (m + (v[..., ci:ci + 1].astype(np.float32) * u[None, None, None, :, :, :, ci].astype(np.float32)))
        m = m.astype(np.float32)
    ho, wo, _, _ = wg.tiles_hw(h, w, pad)
    y = wg.untile(wg.output_transform(m.astype(np.float64)), ho, wo)
    exact = ops.conv2d_fwd(x, f, pad)
    uu = {"f16": 2.0 ** -11, "bf16": 2.0 ** -8}[fmt]
    gam = lambda q: q * 2.0 ** -24 / (1 - q * 2.0 ** -24)  # noqa: E731
    coef = 2 * uu + uu * uu + gam(c) * (1 + uu) ** 2 + gam(9)
    scale = wg.error_scale(x, f, pad)
    assert np.all(np.abs(exact) <= scale * (1 + 1e-12))
    assert np.all(np.abs(y - exact) <= coef * scale)
    # and the bound is not vacuous: the rounding of the transforms shows
    assert np.max(np.abs(y - exact)) > 0.01 * uu * np.max(scale)
