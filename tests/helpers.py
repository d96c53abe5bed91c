"""Helpers shared by the GPU parity tests: moving seeded inputs to the device
and reading results back as exact fp64 values, plus the error metrics."""
from __future__ import annotations

import numpy as np

from oracle.rounding import decode, round_to

DT = {"f32": 0, "f16": 1, "bf16": 2}


def dev(a: np.ndarray, dtype: str):
    """numpy storage array (bf16 as uint16 bits) -> device tensor of that type."""
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    elif dtype == "f16":
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float16))
    elif dtype == "f32":
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    else:
        t = torch.from_numpy(np.ascontiguousarray(a))
    return t.cuda()


def host64(t) -> np.ndarray:
    """device tensor -> exact fp64 values."""
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return decode(t.view(torch.int16).numpy().view(np.uint16), "bf16")
    return t.numpy().astype(np.float64)


def empty(shape, dtype: str):
    import torch
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dtype]
    return torch.empty(tuple(shape), dtype=tdt, device="cuda")


def norm_max_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    """max |gpu - ref| / max |ref| (the parity metric of fp32 outputs)."""
    den = float(np.max(np.abs(ref)))
    return float(np.max(np.abs(gpu - ref))) / (den if den > 0 else 1.0)


def ulp(x: np.ndarray, fmt: str) -> np.ndarray:
    """Spacing of `fmt` numbers at |x| (the subnormal spacing below the normal range)."""
    p, emin = {"f16": (11, -14), "bf16": (8, -126), "f32": (24, -126)}[fmt]
    ax = np.abs(x)
    _, ex = np.frexp(np.where(ax > 0, ax, 1.0))
    e = np.maximum(ex - 1, emin)
    return np.ldexp(1.0, e - (p - 1))


def accum_bound(abs_prod_sum: np.ndarray, k: int) -> np.ndarray:
    """Error bound of an fp32 sum of k products: gamma_k * sum |a_i b_i| with
    gamma_k = k u / (1 - k u), u = 2^-24 (products of fp16/bf16 values are
    exact in fp32)."""
    u = 2.0 ** -24
    return (k * u / (1 - k * u)) * abs_prod_sum


def lowp_close(gpu: np.ndarray, exact: np.ndarray, fmt: str, acc_err=0.0) -> bool:
    """A low-precision output is the storage rounding of a value within
    `acc_err` of the exact result: it may differ from the oracle's rounding of
    the exact value by the accumulation error plus one storage ulp."""
    ref = round_to(exact, fmt)
    both_nan = np.isnan(gpu) & np.isnan(ref)
    d = np.abs(gpu - ref)
    tol = ulp(np.maximum(np.abs(ref), np.abs(gpu)), fmt) + acc_err
    return bool(np.all(both_nan | (d <= tol)))
