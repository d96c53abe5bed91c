"""The SGD update applied inside the weight-gradient product
(mdnn_gemm_tn_update, and the train step's fuse_update built on it).

Section 3.1's update of the fp32 master weights is a pure function of the
stored gradient; doing it in the product's epilogue instead of storing the
gradient and updating from it must give the same weights, momentum and
working copy bit for bit.  So the reference here is the library's own pair
of calls -- the TN product into an fp32 buffer, then mdnn_sgd_update -- on
copies of the same buffers (both are checked against the oracle elsewhere),
for every tile configuration the fused product can take, with and without
momentum and loss scaling, with a scaler whose pending-overflow flag is set
(nothing may change) and with a padded weight matrix (the padding may not
change).  The train step with fuse_update must follow the unfused step's
trajectory bit for bit, forced overflows included.
"""
import dataclasses

import numpy as np
import pytest

import workloads as W
from tests.helpers import DT, dev

pytestmark = pytest.mark.gpu

SHAPES = [  # M, N, K: the pipelined tile the product takes
    (4096, 4096, 1024),   # 256 x 256
    (2048, 4096, 1024),   # 128 x 128, two workgroups per CU
    (1024, 4096, 2048),   # 128 x 128, three stages, one workgroup per CU
    (1024, 1024, 512),    # 64 x 64
]


def _scaler(mdnn, scale, reserved=0):
    """A device scaler; reserved (the pending-overflow flag, the struct's
    eighth 32-bit field) set when asked."""
    import torch
    sc = mdnn.make_scaler(scale)
    if reserved:
        sc.view(torch.int32)[7] = reserved
    return sc


def _operands(m, n, k, dt, seed):
    a = W.normal((k, m), seed, 1, dt, 1.0)
    b = W.normal((k, n), seed, 2, dt, 1.0 / np.sqrt(k))
    return dev(a, dt), dev(b, dt)


def _params(m, ldw, seed, dt):
    import torch
    w = torch.from_numpy(W.normal((m, ldw), seed, 3, "f32", 0.05)).cuda()
    v = torch.from_numpy(W.normal((m, ldw), seed, 4, "f32", 0.01)).cuda()
    lp = w.to(torch.float16 if dt == "f16" else torch.bfloat16)
    return w, v, lp


def _reference(mdnn, A, B, m, n, k, dt, w, v, lp, lr, mom, sc):
    """TN product stored in fp32, then mdnn_sgd_update on copies."""
    import torch
    g = torch.empty((m, n), dtype=torch.float32, device="cuda")
    mdnn.mdnn_gemm_mixed(2, m, n, k, 1.0, A, A.stride(0), B, B.stride(0), DT[dt], 0.0, None, 0, g, n, DT["f32"])
    w, v, lp = w[:, :n].contiguous(), v[:, :n].contiguous(), lp[:, :n].contiguous()
    mdnn.mdnn_sgd_update(m * n, w, g, v if mom else None, lp, DT[dt], lr, mom, sc)
    torch.cuda.synchronize()
    return w, v, lp


@pytest.mark.timeout(300)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "%dx%dx%d" % s)
@pytest.mark.parametrize("mode", ["momentum_scaled", "plain", "momentum", "skipped"])
def test_fused_update_equals_product_then_update(mdnn, shape, mode):
    import torch
    m, n, k = shape
    dt = "bf16" if (mode == "plain" and m == 2048) else "f16"
    A, B = _operands(m, n, k, dt, 7 + m // 1024)
    w, v, lp = _params(m, n, 11, dt)
    lr, mom = (0.01, 0.0) if mode == "plain" else (0.01, 0.9)
    scaled = mode in ("momentum_scaled", "skipped")
    sc_f = _scaler(mdnn, 1024.0, reserved=1 if mode == "skipped" else 0) if scaled else None
    sc_r = _scaler(mdnn, 1024.0, reserved=1 if mode == "skipped" else 0) if scaled else None
    rw, rv, rlp = _reference(mdnn, A, B, m, n, k, dt, w.clone(), v.clone(), lp.clone(), lr, mom, sc_r)
    w0, v0, lp0 = w.clone(), v.clone(), lp.clone()
    mdnn.mdnn_gemm_tn_update(m, n, k, A, A.stride(0), B, B.stride(0), DT[dt], w, v if mom else None, lp, n, lr,
                             mom, sc_f)
    torch.cuda.synchronize()
    assert torch.equal(w, rw) and torch.equal(lp, rlp)
    assert torch.equal(v, rv if mom else v0)
    if mode == "skipped":
        assert torch.equal(w, w0) and torch.equal(v, v0) and torch.equal(lp, lp0)
    else:
        assert not torch.equal(w, w0)
    if scaled:   # only read
        assert torch.equal(sc_f, _scaler(mdnn, 1024.0, reserved=1 if mode == "skipped" else 0))


def test_fused_update_without_working_copy(mdnn):
    """w_lp NULL (no working copy), plain SGD with a loss scaler: the same
    weights as the product stored and mdnn_sgd_update without a copy."""
    import torch
    m, n, k = 1024, 4096, 2048
    A, B = _operands(m, n, k, "f16", 9)
    w, _, _ = _params(m, n, 15, "f16")
    g = torch.empty((m, n), dtype=torch.float32, device="cuda")
    mdnn.mdnn_gemm_mixed(2, m, n, k, 1.0, A, A.stride(0), B, B.stride(0), DT["f16"], 0.0, None, 0, g, n, DT["f32"])
    rw = w.clone()
    mdnn.mdnn_sgd_update(m * n, rw, g, None, None, DT["f16"], 0.03, 0.0, _scaler(mdnn, 512.0))
    mdnn.mdnn_gemm_tn_update(m, n, k, A, A.stride(0), B, B.stride(0), DT["f16"], w, None, None, n, 0.03, 0.0,
                             _scaler(mdnn, 512.0))
    torch.cuda.synchronize()
    assert torch.equal(w, rw)


def test_fused_update_padded_rows(mdnn):
    """ldw > N: the columns past N are never touched."""
    import torch
    m, n, k, ldw = 1024, 1024, 512, 1032
    A, B = _operands(m, n, k, "f16", 5)
    w, v, lp = _params(m, ldw, 13, "f16")
    sc = _scaler(mdnn, 256.0)
    rw, rv, rlp = _reference(mdnn, A, B, m, n, k, "f16", w.clone(), v.clone(), lp.clone(), 0.02, 0.9,
                             _scaler(mdnn, 256.0))
    w0, v0, lp0 = w.clone(), v.clone(), lp.clone()
    mdnn.mdnn_gemm_tn_update(m, n, k, A, A.stride(0), B, B.stride(0), DT["f16"], w, v, lp, ldw, 0.02, 0.9, sc)
    torch.cuda.synchronize()
    assert torch.equal(w[:, :n], rw) and torch.equal(v[:, :n], rv) and torch.equal(lp[:, :n], rlp)
    assert torch.equal(w[:, n:], w0[:, n:]) and torch.equal(v[:, n:], v0[:, n:]) and torch.equal(lp[:, n:], lp0[:, n:])


def test_fused_update_rejects_what_it_cannot_take(mdnn):
    import torch
    A, B = _operands(1024, 1024, 512, "f16", 3)
    w, v, lp = _params(1024, 1024, 3, "f16")

    def call(m=1024, n=1024, k=512, a=A, b=B, dt="f16", ww=w, vv=v, ll=lp, ldw=1024, mom=0.9):
        mdnn.mdnn_gemm_tn_update(m, n, k, a, a.stride(0) if a is not None and a.dim() == 2 else m, b,
                                 b.stride(0) if b is not None and b.dim() == 2 else n, DT[dt], ww, vv, ll, ldw,
                                 0.01, mom, None)

    def status(**kw):
        with pytest.raises(mdnn.MdnnError) as e:
            call(**kw)
        return e.value.status

    assert status(n=1000) == mdnn.ERR_SHAPE            # not a multiple of 256
    assert status(k=500) == mdnn.ERR_SHAPE             # K not whole 64-deep steps
    assert status(m=256, n=256, k=512) == mdnn.ERR_SHAPE   # too few tiles for the pipelined kernel
    assert status(dt="f32") == mdnn.ERR_DTYPE
    assert status(vv=None) == mdnn.ERR_NULL            # momentum needs v32
    assert status(ldw=1000) == mdnn.ERR_LAYOUT
    wf = torch.zeros(1024 * 1024 + 1, dtype=torch.float32, device="cuda")
    assert status(ww=wf[1:]) == mdnn.ERR_MISALIGNED   # w32 only 4-byte aligned
    torch.cuda.synchronize()


def _pair(mdnn, cfg):
    """The same net with and without fuse_update, from the same parameters."""
    params = W.init_params(cfg)
    nets = []
    for fuse in (False, True):
        net = mdnn.Net(cfg.layers, cfg.batch, DT[cfg.dtype], cfg.loss, cfg.lr, cfg.momentum, cfg.loss_scaling,
                       cfg.init_scale, cfg.n_classes, fuse_update=fuse)
        net.set_params(params)
        nets.append(net)
    return nets


def _same_state(mdnn, a, b, n_fused_ranges):
    import torch
    torch.cuda.synchronize()
    assert torch.equal(a.master, b.master)
    if a.mom is not None:
        assert torch.equal(a.mom, b.mom)
    assert torch.equal(a.lowp, b.lowp)
    if a.scaler is not None:
        assert mdnn.read_scaler(a.scaler) == mdnn.read_scaler(b.scaler)
    # the gradients the fused net still stores (all but its fused layers' weights)
    g = torch.ones_like(a.grads, dtype=torch.bool)
    for off, n in n_fused_ranges:
        g[off:off + n] = False
    assert torch.equal(a.grads[g].view(torch.int32), b.grads[g].view(torch.int32))   # bitwise (NaN included)


def _fused_ranges(cfg):
    """Flat (offset, length) of the weights the fused net updates in the
    product: FC layers with in, out multiples of 256, a batch multiple of 64,
    and a product of at least 128 tiles of 128 x 128 (so that the unfused
    step does not split it over K)."""
    out, off = [], 0
    for i, l in enumerate(cfg.layers):
        nw = l.c_in * l.c_out
        if (l.c_in % 256 == 0 and l.c_out % 256 == 0 and cfg.batch % 64 == 0
                and (l.c_in // 128) * (l.c_out // 128) >= 128):
            out.append((off, nw))
        off += nw + l.c_out
    return out


@pytest.mark.timeout(300)
@pytest.mark.parametrize("case", ["scaled_with_overflows", "input_beyond_fp16", "bf16_unscaled", "full_size"])
def test_train_step_fused_matches_unfused(mdnn, case):
    """fuse_update changes where the update of the hidden layers' weights
    runs, not what it computes: the trajectories agree bit for bit (loss,
    master weights, momentum, working copy, scaler state, stored gradients),
    here through steps whose update is skipped (initial scale 2^40: the
    scaled gradients overflow in fp16 until the scale has halved enough) and
    the applied steps after them, through an input value that overflows
    fp16 when the batch is stored (only the input cast can see it before the
    first layer's fused product runs), with bf16 storage and no loss scaling
    (the only way bf16 nets fuse), and at the benchmark's full size."""
    import torch
    if case == "full_size":
        cfg, steps = W.wide_mlp_fp16(), 4
    elif case == "input_beyond_fp16":
        cfg, steps = W.wide_mlp_fp16(batch=512, width=2048), 3
    elif case == "bf16_unscaled":   # bf16 storage fuses only without loss scaling
        cfg, steps = dataclasses.replace(W.wide_mlp_fp16(batch=512, width=2048), dtype="bf16",
                                         loss_scaling=False), 3
    else:
        cfg, steps = W.wide_mlp_fp16(batch=512, width=2048, init_scale=2.0 ** 40), 30
    fr = _fused_ranges(cfg)
    assert fr, "the case is meant to fuse"
    plain, fused = _pair(mdnn, cfg)
    skipped = 0
    for s in range(steps):
        x, t = W.batch_inputs(cfg, s)
        if case == "input_beyond_fp16" and s == 1:
            x[5, 7] = 1.0e6   # finite in fp32, Inf once stored in fp16: the step must skip its update
        X, T = dev(x, "f32"), dev(t, "f32")
        la = plain.step(X, T)
        lb = fused.step(X, T)
        assert torch.equal(la.view(torch.int32), lb.view(torch.int32)), f"step {s}"   # bitwise (NaN included)
        _same_state(mdnn, plain, fused, fr)
        if fused.scaler is None:
            continue
        skipped += mdnn.read_scaler(fused.scaler)["overflow"]
        if case == "input_beyond_fp16":
            assert mdnn.read_scaler(fused.scaler)["overflow"] == (1 if s == 1 else 0), f"step {s}"
    if case in ("scaled_with_overflows", "input_beyond_fp16"):
        assert skipped >= 1, "the case is meant to skip updates"
    if fused.scaler is not None:
        assert mdnn.read_scaler(fused.scaler)["good_steps"] >= 1
