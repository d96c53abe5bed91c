"""Pins of the oracle's storage rounding against library conversions.

The definition (``round_generic``) is pinned to numpy's IEEE conversions for
fp16 and fp32 (round to nearest even, straight from fp64) and to torch's CPU
bfloat16 conversion of fp32 values; the fast ``round_to`` is pinned to the
definition and to the same libraries.  The sets include every representable
value, every tie between neighbours, values one fp64/fp32 ulp either side of
each tie, subnormals, overflow and NaN.
"""
import math

import numpy as np
import pytest

from oracle.rounding import decode, encode, max_finite, round_generic, round_to

BOTH = pytest.mark.parametrize("rnd", [round_generic, round_to], ids=["generic", "fast"])


def _all_f16():
    v = np.arange(65536, dtype=np.uint32).astype(np.uint16).view(np.float16).astype(np.float64)
    return v[np.isfinite(v)]


@BOTH
def test_f16_exhaustive_values_and_ties(rnd):
    v = np.unique(_all_f16())
    assert np.array_equal(rnd(v, "f16"), v)
    mids = (v[:-1] + v[1:]) / 2.0                 # exact in fp64
    probes = np.concatenate([mids, np.nextafter(mids, np.inf), np.nextafter(mids, -np.inf)])
    with np.errstate(over="ignore"):
        want = probes.astype(np.float16).astype(np.float64)
    got = rnd(probes, "f16")
    assert np.array_equal(got, want)


@BOTH
def test_f16_overflow_subnormal_nan(rnd):
    big = max_finite("f16")
    assert big == 65504.0
    half_ulp = 16.0
    x = np.array([big + half_ulp - 1e-9, big + half_ulp, 1e5, -1e5, 2.0 ** -25, 3 * 2.0 ** -25,
                  2.0 ** -24, 2.0 ** -26, np.inf, -np.inf])
    got = rnd(x, "f16")
    assert got[0] == big and got[1] == np.inf and got[2] == np.inf and got[3] == -np.inf
    assert got[4] == 0.0 and got[5] == 2.0 ** -23 and got[6] == 2.0 ** -24 and got[7] == 0.0
    assert np.isinf(got[8]) and np.isinf(got[9])
    assert np.isnan(rnd(np.array([np.nan]), "f16"))[0]
    # negative zero and sign symmetry
    assert math.copysign(1.0, rnd(np.array([-2.0 ** -30]), "f16")[0]) == -1.0


@BOTH
def test_f16_random_wide_range(rnd):
    g = np.random.default_rng(7)
    x = g.standard_normal(400_000) * np.exp2(g.integers(-30, 20, 400_000))
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).astype(np.float64)
    assert np.array_equal(rnd(x, "f16"), want)


@BOTH
def test_f32_against_numpy(rnd):
    g = np.random.default_rng(8)
    x = g.standard_normal(400_000) * np.exp2(g.integers(-160, 130, 400_000))
    with np.errstate(over="ignore"):
        want = x.astype(np.float32).astype(np.float64)
    assert np.array_equal(rnd(x, "f32"), want)


def _torch_bf16(x32: np.ndarray) -> np.ndarray:
    torch = pytest.importorskip("torch")
    return torch.from_numpy(x32.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


@BOTH
def test_bf16_against_torch_all_values_and_ties(rnd):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = decode(bits, "bf16")
    v = np.unique(v[np.isfinite(v)])
    assert np.array_equal(rnd(v, "bf16"), v)
    mids = (v[:-1] + v[1:]) / 2.0                 # 9 significant bits: exact in fp32
    m32 = mids.astype(np.float32)
    assert np.array_equal(m32.astype(np.float64), mids)
    probes = np.concatenate([m32, np.nextafter(m32, np.float32(np.inf)),
                             np.nextafter(m32, np.float32(-np.inf))]).astype(np.float64)
    assert np.array_equal(rnd(probes, "bf16"), _torch_bf16(probes))


@BOTH
def test_bf16_random_fp32_inputs(rnd):
    g = np.random.default_rng(9)
    x = (g.standard_normal(400_000) * np.exp2(g.integers(-140, 128, 400_000))).astype(np.float32)
    x = x[np.isfinite(x)].astype(np.float64)
    assert np.array_equal(rnd(x, "bf16"), _torch_bf16(x))


@BOTH
def test_bf16_keeps_fp32_range_fp16_does_not(rnd):
    """Section 3.2: bfloat16 has fp32's range, so converting fp32 data to it does
    not overflow or underflow for lack of exponent range; fp16 does."""
    x = np.array([1e38, -3.0e38, 2.0 ** -126, 1e-38])
    b = rnd(x, "bf16")
    assert np.all(np.isfinite(b)) and np.all(b != 0.0)
    h = rnd(x, "f16")
    assert np.isinf(h[0]) and np.isinf(h[1]) and h[2] == 0.0 and h[3] == 0.0


def test_encode_decode_roundtrip():
    g = np.random.default_rng(10)
    x = g.standard_normal(1000)
    for fmt in ("f16", "bf16", "f32"):
        r = round_to(x, fmt)
        assert np.array_equal(decode(encode(r, fmt), fmt), r)


def test_fast_bf16_matches_definition_everywhere():
    g = np.random.default_rng(11)
    x = g.standard_normal(1_000_000) * np.exp2(g.integers(-140, 129, 1_000_000))
    x = np.concatenate([x, [np.inf, -np.inf, 0.0, -0.0, max_finite("bf16"), 3.3961e38, 3.4e38,
                            2.0 ** -126, 2.0 ** -127, 2.0 ** -133, 2.0 ** -134, 1.5 * 2.0 ** -133]])
    with np.errstate(over="ignore"):
        a, b = round_to(x, "bf16"), round_generic(x, "bf16")
    assert np.array_equal(a, b)
    assert np.isnan(round_to(np.array([np.nan]), "bf16"))[0]
