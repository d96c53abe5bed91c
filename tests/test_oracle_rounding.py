"""Pins of the oracle's storage rounding against library conversions.

fp16 and fp32 are pinned to numpy's IEEE conversions (round to nearest even,
straight from fp64); bf16 to torch's CPU bfloat16 conversion of fp32 values.
The sets include every representable value, every tie between neighbours,
values one fp64/fp32 ulp either side of each tie, subnormals, overflow and NaN.
"""
import math

import numpy as np
import pytest

from oracle.rounding import round_to, decode, encode, max_finite


def _all_f16():
    v = np.arange(65536, dtype=np.uint32).astype(np.uint16).view(np.float16).astype(np.float64)
    return v[np.isfinite(v)]


def test_f16_exhaustive_values_and_ties():
    v = np.unique(_all_f16())
    assert np.array_equal(round_to(v, "f16"), v)
    mids = (v[:-1] + v[1:]) / 2.0                 # exact in fp64
    probes = np.concatenate([mids, np.nextafter(mids, np.inf), np.nextafter(mids, -np.inf)])
    with np.errstate(over="ignore"):
        want = probes.astype(np.float16).astype(np.float64)
    got = round_to(probes, "f16")
    assert np.array_equal(got, want)


def test_f16_overflow_subnormal_nan():
    big = max_finite("f16")
    assert big == 65504.0
    half_ulp = 16.0
    x = np.array([big + half_ulp - 1e-9, big + half_ulp, 1e5, -1e5, 2.0 ** -25, 3 * 2.0 ** -25,
                  2.0 ** -24, 2.0 ** -26, np.inf, -np.inf])
    got = round_to(x, "f16")
    assert got[0] == big and got[1] == np.inf and got[2] == np.inf and got[3] == -np.inf
    assert got[4] == 0.0 and got[5] == 2.0 ** -23 and got[6] == 2.0 ** -24 and got[7] == 0.0
    assert np.isinf(got[8]) and np.isinf(got[9])
    assert np.isnan(round_to(np.array([np.nan]), "f16"))[0]
    # negative zero and sign symmetry
    assert math.copysign(1.0, round_to(np.array([-2.0 ** -30]), "f16")[0]) == -1.0


def test_f16_random_wide_range():
    g = np.random.default_rng(7)
    x = g.standard_normal(400_000) * np.exp2(g.integers(-30, 20, 400_000))
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).astype(np.float64)
    assert np.array_equal(round_to(x, "f16"), want)


def test_f32_against_numpy():
    g = np.random.default_rng(8)
    x = g.standard_normal(400_000) * np.exp2(g.integers(-160, 130, 400_000))
    with np.errstate(over="ignore"):
        want = x.astype(np.float32).astype(np.float64)
    assert np.array_equal(round_to(x, "f32"), want)


def _torch_bf16(x32: np.ndarray) -> np.ndarray:
    torch = pytest.importorskip("torch")
    return torch.from_numpy(x32.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


def test_bf16_against_torch_all_values_and_ties():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = decode(bits, "bf16")
    v = np.unique(v[np.isfinite(v)])
    assert np.array_equal(round_to(v, "bf16"), v)
    mids = (v[:-1] + v[1:]) / 2.0                 # 9 significant bits: exact in fp32
    m32 = mids.astype(np.float32)
    assert np.array_equal(m32.astype(np.float64), mids)
    probes = np.concatenate([m32, np.nextafter(m32, np.float32(np.inf)),
                             np.nextafter(m32, np.float32(-np.inf))]).astype(np.float64)
    assert np.array_equal(round_to(probes, "bf16"), _torch_bf16(probes))


def test_bf16_random_fp32_inputs():
    g = np.random.default_rng(9)
    x = (g.standard_normal(400_000) * np.exp2(g.integers(-140, 128, 400_000))).astype(np.float32)
    x = x[np.isfinite(x)].astype(np.float64)
    assert np.array_equal(round_to(x, "bf16"), _torch_bf16(x))


def test_bf16_keeps_fp32_range_fp16_does_not():
    """Section 3.2: bfloat16 has fp32's range, so converting fp32 data to it does
    not overflow or underflow for lack of exponent range; fp16 does."""
    x = np.array([1e38, -3.0e38, 2.0 ** -126, 1e-38])
    b = round_to(x, "bf16")
    assert np.all(np.isfinite(b)) and np.all(b != 0.0)
    h = round_to(x, "f16")
    assert np.isinf(h[0]) and np.isinf(h[1]) and h[2] == 0.0 and h[3] == 0.0


def test_encode_decode_roundtrip():
    g = np.random.default_rng(10)
    x = g.standard_normal(1000)
    for fmt in ("f16", "bf16", "f32"):
        r = round_to(x, fmt)
        assert np.array_equal(decode(encode(r, fmt), fmt), r)
