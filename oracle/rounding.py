"""Round-to-nearest-even storage rounding, written from the IEEE-754 definition.

Section 3.2 of the paper names the two 16-bit formats the step stores in:
IEEE half precision (fp16: 11 significand bits, exponents -14..15) and
bfloat16 (8 significand bits with fp32's exponent range -126..127, so that
converting fp32 data to it cannot overflow or underflow for lack of range).

``round_generic(x, fmt)`` is the definition: the nearest ``fmt`` number, ties
to even, with gradual underflow (subnormals kept), overflow to +-inf and NaN
kept NaN, rounded *directly* from fp64 (one rounding).

``round_to(x, fmt)`` computes the same function faster: numpy's IEEE
conversions for fp16 and fp32 (library routines), and for bfloat16 the
round-half-even rule applied to the fp64 bit pattern (add half an ulp minus
one plus the kept lowest bit, then truncate) wherever the result is a normal
number, the definition elsewhere.  Tests pin both against each other and
against numpy / torch conversions.

Test infrastructure only (see the package header).
"""
from __future__ import annotations

import numpy as np

# name -> (significand bits incl. the implicit one, emin, emax)
FORMATS = {
    "f16": (11, -14, 15),
    "bf16": (8, -126, 127),
    "f32": (24, -126, 127),
    "f64": None,
}


def max_finite(fmt: str) -> float:
    p, _, emax = FORMATS[fmt]
    return (2.0 - 2.0 ** (1 - p)) * 2.0 ** emax


def round_generic(x, fmt: str) -> np.ndarray:
    """Nearest ``fmt`` value of each fp64 element, ties to even (definition)."""
    x = np.asarray(x, dtype=np.float64)
    if fmt == "f64":
        return x.copy()
    p, emin, emax = FORMATS[fmt]
    out = x.copy()
    sel = np.isfinite(x) & (x != 0.0)
    ax = np.abs(x[sel])
    _, ex = np.frexp(ax)              # ax = m * 2**ex, m in [0.5, 1)
    e = np.maximum(ex - 1, emin)      # ax in [2**e, 2**(e+1)); subnormal range uses emin
    q = np.ldexp(1.0, e - (p - 1))    # spacing of fmt numbers in that binade
    r = np.round(ax / q) * q          # np.round: halves to even; ax/q is exact
    r = np.where(r > max_finite(fmt), np.inf, r)
    out[sel] = np.copysign(r, x[sel])
    return out


_BF16_DROP = 52 - 7                   # fp64 fraction bits below bfloat16's 7
_BF16_MIN_NORMAL = 2.0 ** -126


def _round_bf16(x: np.ndarray) -> np.ndarray:
    u = x.view(np.uint64)
    lsb = (u >> np.uint64(_BF16_DROP)) & np.uint64(1)
    r = (u + (np.uint64((1 << (_BF16_DROP - 1)) - 1) + lsb)) & \
        ~np.uint64((1 << _BF16_DROP) - 1)
    out = r.view(np.float64)
    ax = np.abs(x)
    out = np.where(np.abs(out) > max_finite("bf16"), np.copysign(np.inf, x), out)
    out = np.where(np.isnan(x), x, out)
    small = (ax < _BF16_MIN_NORMAL) & (ax != 0.0)
    if np.any(small):
        out[small] = round_generic(x[small], "bf16")
    return out


def round_to(x, fmt: str) -> np.ndarray:
    """Nearest ``fmt`` value of each fp64 element, ties to even."""
    x = np.asarray(x, dtype=np.float64)
    if fmt == "f64":
        return x.copy()
    with np.errstate(over="ignore", invalid="ignore"):
        if fmt == "f32":
            return x.astype(np.float32).astype(np.float64)
        if fmt == "f16":
            return x.astype(np.float16).astype(np.float64)
    if fmt == "bf16":
        return _round_bf16(np.ascontiguousarray(x))
    raise ValueError(fmt)


def decode(a: np.ndarray, fmt: str) -> np.ndarray:
    """Exact fp64 value of stored elements (bf16 given as uint16 bit patterns)."""
    a = np.asarray(a)
    if fmt == "bf16":
        if a.dtype != np.uint16:
            raise TypeError("bf16 data must be uint16 bit patterns")
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def encode(x: np.ndarray, fmt: str) -> np.ndarray:
    """Storage bits of values that are already ``fmt`` numbers (no rounding)."""
    x = np.asarray(x, dtype=np.float64)
    if fmt == "f16":
        return x.astype(np.float16)
    if fmt == "f32":
        return x.astype(np.float32)
    if fmt == "bf16":
        return (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    raise ValueError(fmt)
