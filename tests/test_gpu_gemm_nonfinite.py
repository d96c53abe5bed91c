"""The overflow flag of mdnn_gemm_mixed_ws (nonfinite): the dynamic loss
scaler's test that every stored gradient is finite, done by the GEMM that
stores it instead of by a second pass over the gradient buffer.

For each kernel path an fp32 output can take -- the 256 x 256 and 128 x 128
pipelined kernels (two and four LDS stages), the split-K reduction, the
general MFMA kernel, the skinny rows / cols / depth kernels, the fp32 kernel
-- a single Inf planted in A makes a whole row of D non-finite and must set
the flag; the same product with finite inputs must leave it at 0 and store
exactly what the call without the flag stores.  The flag is never cleared by
the library.  16-bit outputs are tested on the stored values (a finite
result that rounds to Inf counts).  The planted value and the all-finite expectation come from the
inputs alone (Inf times a nonzero finite value is not finite), no oracle
arithmetic is needed.
"""
import numpy as np
import pytest

import workloads as W
from tests.helpers import DT, dev

pytestmark = pytest.mark.gpu

LAYOUT = {"NN": 0, "NT": 1, "TN": 2}
CASES = [  # layout, m, n, k, ab dtype, workspace: which path
    ("TN", 4096, 4096, 64, "f16", False),   # 256 x 256 pipelined kernel
    ("NN", 3072, 3072, 64, "f16", False),   # 128 x 128, two stages (more tiles than CUs)
    ("NT", 1024, 1024, 128, "bf16", False),  # 128 x 128, four stages (one workgroup per CU)
    ("TN", 256, 256, 4096, "f16", True),    # split K over the workspace, reduction epilogue
    ("NN", 200, 136, 100, "f16", False),    # K % 64 != 0: general MFMA kernel
    ("NN", 4096, 1, 4096, "f16", False),    # skinny rows (regression head)
    ("TN", 4096, 1, 4096, "f16", True),     # skinny cols, split over the workspace
    ("TN", 512, 1, 16, "bf16", False),      # skinny cols, one pass
    ("NT", 1024, 1024, 1, "f16", False),    # skinny depth (K = 1 outer product)
    ("NN", 300, 200, 150, "f32", False),    # fp32 kernel
    ("TN", 64, 128, 4096, "f32", True),     # fp32 split K
]


def _call(mdnn, layout, A, B, m, n, k, ws, flag):
    import torch
    D = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
    args = (LAYOUT[layout], m, n, k, 1.0, A, A.stride(0), B, B.stride(0), mdnn.dtype_of(A), 0.0, None, 0,
            D, D.stride(0), DT["f32"], None, 0, None, 0)
    mdnn.mdnn_gemm_mixed_ws(*args, ws, ws.numel() if ws is not None else 0, nonfinite=flag)
    torch.cuda.synchronize()
    return D


@pytest.mark.parametrize("case", CASES, ids=lambda c: "%s_%dx%dx%d_%s%s" % (c[0], c[1], c[2], c[3], c[4],
                                                                            "_ws" if c[5] else ""))
def test_flag_set_exactly_when_a_stored_value_is_not_finite(mdnn, case):
    import torch
    layout, m, n, k, dt, use_ws = case
    sa = (k, m) if layout == "TN" else (m, k)
    sb = (n, k) if layout == "NT" else (k, n)
    a = W.normal(sa, 61, 1, dt, 1 / np.sqrt(k))
    b = W.normal(sb, 61, 2, dt)
    ws = None
    if use_ws:
        nb = mdnn.mdnn_gemm_workspace(DT[dt], m, n, k)
        assert nb > 0, "the case is meant to split"
        ws = torch.empty((nb,), dtype=torch.uint8, device="cuda")
    A, B = dev(a, dt), dev(b, dt)
    flag = torch.zeros((1,), dtype=torch.int32, device="cuda")
    plain = _call(mdnn, layout, A, B, m, n, k, ws, None)
    checked = _call(mdnn, layout, A, B, m, n, k, ws, flag)
    assert torch.isfinite(plain).all()
    assert torch.equal(plain, checked)
    assert int(flag.item()) == 0
    # one Inf in A: row 7 of D (A[7][0], or A[0][7] stored transposed)
    A[(0, 7) if layout == "TN" else (7, 0)] = float("inf")
    got = _call(mdnn, layout, A, B, m, n, k, ws, flag)
    assert not torch.isfinite(got[7]).any()
    assert int(flag.item()) == 1
    # never cleared: a finite product leaves a set flag set
    A[(0, 7) if layout == "TN" else (7, 0)] = 0.0
    _call(mdnn, layout, A, B, m, n, k, ws, flag)
    assert int(flag.item()) == 1


CASES16 = [  # layout, m, n, k, dtype of A, B and D: which path
    ("NN", 4096, 4096, 64, "f16"),    # 256 x 256 pipelined kernel
    ("NT", 1024, 1024, 128, "bf16"),  # 128 x 128 pipelined kernel
    ("NN", 200, 136, 100, "f16"),     # general MFMA kernel
    ("NT", 1024, 1024, 1, "f16"),     # skinny depth (outer product)
]


@pytest.mark.parametrize("case", CASES16, ids=lambda c: "%s_%dx%dx%d_%s" % c)
def test_flag_on_16bit_outputs(mdnn, case):
    """A 16-bit D is tested as stored: Inf planted in A sets the flag, and so
    does (fp16) a finite fp32 result that rounds to Inf -- the same row stored
    in fp32 stays finite and leaves a fresh flag at 0."""
    import torch
    layout, m, n, k, dt = case
    sa = (m, k)
    sb = (n, k) if layout == "NT" else (k, n)
    a = W.normal(sa, 62, 1, dt, 1.0)
    b = W.normal(sb, 62, 2, dt, 1 / np.sqrt(k))
    A, B = dev(a, dt), dev(b, dt)
    tdt = torch.float16 if dt == "f16" else torch.bfloat16

    def run(flag, out=dt):
        D = torch.zeros((m, n), dtype=tdt if out != "f32" else torch.float32, device="cuda")
        mdnn.mdnn_gemm_mixed_ws(LAYOUT[layout], m, n, k, 1.0, A, A.stride(0), B, B.stride(0), DT[dt], 0.0, None,
                                0, D, n, DT[out], None, 0, None, 0, None, 0, nonfinite=flag)
        torch.cuda.synchronize()
        return D

    flag = torch.zeros((1,), dtype=torch.int32, device="cuda")
    assert torch.equal(run(None), run(flag)) and int(flag.item()) == 0
    A[7, 0] = float("inf")
    got = run(flag)
    assert not torch.isfinite(got[7]).any() and int(flag.item()) == 1
    if dt == "f16":
        A[7, :] = 60000.0   # finite, but row 7 of the product is far beyond fp16's range
        flag.zero_()
        got = run(flag)
        assert not torch.isfinite(got[7]).all() and int(flag.item()) == 1
        f32 = torch.zeros((1,), dtype=torch.int32, device="cuda")
        assert torch.isfinite(run(f32, "f32")).all() and int(f32.item()) == 0
