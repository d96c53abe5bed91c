"""GPU parity of mdnn_train_step (forward, loss, backpropagation, SGD update)
against the oracle's step on the same seeded inputs.

The gate: the loss of every step (the forward loss before that step's
update) within 1e-3 relative of the oracle's, over 10 steps (MLP fp32 and
LeNet bf16 and the loss-scaled fp16 wide MLP at their full sizes, the wide
MLP also at reduced width).  Also: every layer's stored
output inside the step, reproducibility (bitwise-identical reruns), dynamic loss scaling
through a forced overflow, and master weights after the run.
"""
import numpy as np
import pytest

import workloads as W
from oracle import train
from tests.helpers import DT, dev, norm_max_err

pytestmark = pytest.mark.gpu
REL = 1e-3


def _gpu_net(mdnn, cfg, params=None):
    net = mdnn.Net(cfg.layers, cfg.batch, DT[cfg.dtype], cfg.loss, cfg.lr, cfg.momentum,
                   cfg.loss_scaling, cfg.init_scale, cfg.n_classes)
    net.set_params(W.init_params(cfg) if params is None else params)
    return net


def _target(cfg, t):
    return dev(t, "f32") if cfg.loss == W.LOSS_MSE else dev(t, "i32")


def _trajectory(mdnn, cfg, steps, params=None):
    net = _gpu_net(mdnn, cfg, params)
    losses = []
    for s in range(steps):
        x, t = W.batch_inputs(cfg, s)
        losses.append(float(net.step(dev(x, "f32"), _target(cfg, t)).item()))
    return losses, net


def _oracle_trajectory(cfg, steps, params=None):
    orc = train.from_config(cfg, W.init_params(cfg) if params is None else params)
    losses = []
    for s in range(steps):
        x, t = W.batch_inputs(cfg, s)
        losses.append(orc.step(x, t))
    return losses, orc


def _check(gl, ol):
    for s, (g, o) in enumerate(zip(gl, ol)):
        assert abs(g - o) <= REL * abs(o), f"step {s}: gpu {g} oracle {o} (all: {gl} vs {ol})"


def test_mlp784_fp32_ten_steps(mdnn):
    cfg = W.mlp784_fp32()
    gl, net = _trajectory(mdnn, cfg, 10)
    ol, orc = _oracle_trajectory(cfg, 10)
    _check(gl, ol)
    w = net.master.cpu().numpy().astype(np.float64)
    assert norm_max_err(w, orc.w32) <= 1e-4


@pytest.mark.timeout(300)
def test_lenet_bf16_ten_steps(mdnn):
    cfg = W.lenet_bf16()
    gl, net = _trajectory(mdnn, cfg, 10)
    ol, orc = _oracle_trajectory(cfg, 10)
    _check(gl, ol)
    assert gl[-1] < gl[0]
    w = net.master.cpu().numpy().astype(np.float64)
    assert norm_max_err(w, orc.w32) <= 1e-3


def test_deep_conv_net_ten_steps(mdnn):
    """Six 3x3 convolution layers (batch 32, 16x16, 8 channels; every layer's
    weight and bias sums take the many-splits second pass, more of them than
    one batched launch holds) and a classifier: losses and master weights
    against the oracle."""
    convs = [W.Layer(W.CONV, 1 if i == 0 else 8, 16, 16, 8, 3, 3, 1, W.ACT_RELU) for i in range(6)]
    cfg = W.TrainConfig(name="deep_conv_bf16_b32", base_seed=1188 + 41,
                        layers=tuple(convs) + (W.Layer(W.FC, 16 * 16 * 8, c_out=10),),
                        batch=32, in_features=256, dtype="bf16", loss=W.LOSS_XENT, lr=0.01)
    gl, net = _trajectory(mdnn, cfg, 10)
    ol, orc = _oracle_trajectory(cfg, 10)
    _check(gl, ol)
    w = net.master.cpu().numpy().astype(np.float64)
    assert norm_max_err(w, orc.w32) <= 1e-3


@pytest.mark.timeout(300)
def test_wide_mlp_fp16_reduced_ten_steps(mdnn):
    cfg = W.wide_mlp_fp16(batch=512, width=1024)
    gl, net = _trajectory(mdnn, cfg, 10)
    ol, orc = _oracle_trajectory(cfg, 10)
    _check(gl, ol)
    s = mdnn.read_scaler(net.scaler)
    assert s["scale"] == orc.scaler["scale"] and s["good_steps"] == orc.scaler["good_steps"]
    w = net.master.cpu().numpy().astype(np.float64)
    assert norm_max_err(w, orc.w32) <= 1e-3


@pytest.mark.timeout(600)
def test_wide_mlp_fp16_full_size_ten_steps(mdnn):
    """The full wide MLP (batch 4096, 4 x 4096 hidden), as the benchmark runs
    it, for the ten steps of the trajectory gate; then the loss scaler's state
    and the fp32 master weights against the oracle's."""
    cfg = W.wide_mlp_fp16()
    gl, net = _trajectory(mdnn, cfg, 10)
    ol, orc = _oracle_trajectory(cfg, 10)
    _check(gl, ol)
    s = mdnn.read_scaler(net.scaler)
    assert s["scale"] == orc.scaler["scale"] and s["good_steps"] == orc.scaler["good_steps"] == 10
    w = net.master.cpu().numpy().astype(np.float64)
    assert norm_max_err(w, orc.w32) <= 1e-3


@pytest.mark.timeout(300)
def test_wide_mlp_full_size_trains_without_skipped_updates(mdnn):
    """The benchmark's workload over 60 steps cycling over 10 batches (as the
    benchmark feeds it): no step overflows (every update is applied, the
    scale stays 2^16) and the loss falls well below its start."""
    import torch
    cfg = W.wide_mlp_fp16()
    net = _gpu_net(mdnn, cfg)
    dev_b = []
    for s in range(10):
        x, t = W.batch_inputs(cfg, s)
        dev_b.append((dev(x, "f32"), _target(cfg, t)))
    losses = torch.zeros(60, device="cuda")
    for i in range(60):
        net.step(*dev_b[i % 10], loss_out=losses[i:i + 1])
    ls = losses.cpu().numpy()
    sc = mdnn.read_scaler(net.scaler)
    assert sc["good_steps"] == 60 and sc["scale"] == 2.0 ** 16 and sc["overflow"] == 0
    assert np.all(np.isfinite(ls)) and ls[-10:].mean() < 0.5 * ls[0], ls


def test_forced_overflow_skips_steps(mdnn):
    """Initial loss scale 2^40: the scaled fp16 loss gradient overflows, the
    update is skipped and the scale halves until it fits; the trajectory
    (skipped steps included) matches the oracle's."""
    cfg = W.wide_mlp_fp16(batch=256, width=256, init_scale=2.0 ** 40)
    gl, net = _trajectory(mdnn, cfg, 6)
    ol, orc = _oracle_trajectory(cfg, 6)
    _check(gl, ol)
    s = mdnn.read_scaler(net.scaler)
    assert s["scale"] == orc.scaler["scale"] < 2.0 ** 40
    assert s["good_steps"] == orc.scaler["good_steps"]


def _stored(net, i, n, dt):
    """Activation i of the last forward pass, read from the bound workspace."""
    import torch
    nbytes = n * (4 if dt == torch.float32 else 2)
    off = net.activation_ptr(i) - net.ws.data_ptr()
    return net.ws[off:off + nbytes].clone().view(dt)


def test_layer_outputs_inside_the_step(mdnn):
    """Each stored activation of the first forward pass of the LeNet chain
    against the oracle's layer applied to the GPU's own stored input of that
    layer (same bits in, so the per-op bar applies inside the chain)."""
    import torch
    from oracle import ops
    from oracle.rounding import round_to
    from tests.helpers import accum_bound, lowp_close
    cfg = W.lenet_bf16()
    p = W.init_params(cfg)
    net = _gpu_net(mdnn, cfg, p)
    x, t = W.batch_inputs(cfg, 0)
    net.step(dev(x, "f32"), _target(cfg, t))
    torch.cuda.synchronize()
    B = cfg.batch
    wl = round_to(p.astype(np.float64), "bf16")
    a0 = _stored(net, 0, B * cfg.in_features, torch.bfloat16).float().cpu().numpy().astype(np.float64)
    assert np.array_equal(a0, round_to(x.astype(np.float64), "bf16").reshape(-1))
    for i, (l, (wo, bo)) in enumerate(zip(cfg.layers, cfg.param_offsets())):
        last = i == len(cfg.layers) - 1
        dt = torch.float32 if last else torch.bfloat16
        a_in = _stored(net, i, B * l.c_in * l.h * l.w, torch.bfloat16).float().cpu().numpy().astype(np.float64)
        got = _stored(net, i + 1, B * l.out_features(), dt).float().cpu().numpy().astype(np.float64)
        b = p[bo:bo + l.n_bias].astype(np.float64)
        if l.kind == W.FC:
            w = wl[wo:wo + l.n_weight].reshape(l.c_in, l.c_out)
            a2 = a_in.reshape(B, -1)
            z = a2 @ w + b
            bound = accum_bound(np.abs(a2) @ np.abs(w) + np.abs(b), l.c_in + 1)
        elif l.kind == W.CONV:
            w = wl[wo:wo + l.n_weight].reshape(l.c_out, l.r, l.s, l.c_in)
            a4 = a_in.reshape(B, l.h, l.w, l.c_in)
            z = ops.conv2d_fwd(a4, w, l.pad) + b
            bound = accum_bound(ops.conv2d_fwd(np.abs(a4), np.abs(w), l.pad) + np.abs(b),
                                l.r * l.s * l.c_in + 1)
        else:
            y, _ = ops.maxpool2_fwd(a_in.reshape(B, l.h, l.w, l.c_in))
            assert np.array_equal(got, y.reshape(-1)), i
            continue
        if l.act == W.ACT_RELU:
            z = ops.relu(z)
        if last:
            assert norm_max_err(got, z.reshape(-1)) <= 1e-4, i
        else:
            assert lowp_close(got, z.reshape(-1), "bf16", bound.reshape(-1)), i


def test_train_step_reproducible(mdnn):
    cfg = W.lenet_bf16()
    gl1, n1 = _trajectory(mdnn, cfg, 3)
    gl2, n2 = _trajectory(mdnn, cfg, 3)
    assert gl1 == gl2
    assert bool((n1.master == n2.master).all()) and bool((n1.lowp == n2.lowp).all())


@pytest.mark.timeout(300)
@pytest.mark.parametrize("size", [(512, 1024, "f16"), (4096, 4096, "f16"), (100, 512, "bf16")],
                         ids=["b512_w1024", "full_b4096_w4096", "b100_w512_bf16"])
def test_wide_mlp_first_layer_gradients_from_stored_values(mdnn, size):
    """Weight and bias gradients of the two first layers after one loss-scaled
    step, against their definitions (dW = X^T dZ, db = column sums of dZ)
    evaluated in fp64 on the GPU's own stored X and dZ (the same bits in, so a
    rounding difference earlier in the chain -- a ReLU mask decided the other
    way -- cannot show up here); bar: fp32 accumulation of B exact products,
    gamma_B * sum |terms|.  In this step the weight-gradient GEMMs carry the
    overflow test in their epilogue (256x256 tiles at full size, split K over
    the workspace at width 1024) and the bias gradients' column sums are
    finished for all layers, with the overflow test, in one pass.  Also: the
    stored dZ of layer 0 is zero wherever the layer's ReLU output is not
    positive.  The bias sums read the 16-bit dZ in 64-row chunks of whole
    rows; batch 100 leaves a ragged chunk of 36 rows."""
    import dataclasses
    import torch
    from tests.helpers import accum_bound
    batch, width, dt = size
    cfg = dataclasses.replace(W.wide_mlp_fp16(batch=batch, width=width), dtype=dt)
    net = _gpu_net(mdnn, cfg)
    x, t = W.batch_inputs(cfg, 0)
    net.step(dev(x, "f32"), _target(cfg, t))
    torch.cuda.synchronize()
    g = net.grads.cpu().numpy().astype(np.float64)
    L = len(cfg.layers)

    def stored(ptr, n):
        off = ptr - net.ws.data_ptr()
        st = torch.float16 if dt == "f16" else torch.bfloat16
        return net.ws[off:off + 2 * n].clone().view(st).float().cpu().numpy().astype(np.float64)

    dz = {}
    for i, (wo, bo) in enumerate(cfg.param_offsets()[:2]):
        l = cfg.layers[i]
        a = stored(net.activation_ptr(i), batch * l.c_in).reshape(batch, l.c_in)
        d = stored(net.output_grad_ptr((L - 1 - i) % 2), batch * l.c_out).reshape(batch, l.c_out)
        dz[i] = d
        dw = g[wo:wo + l.c_in * l.c_out].reshape(l.c_in, l.c_out)
        db = g[bo:bo + l.c_out]
        assert np.all(np.abs(dw - a.T @ d) <= accum_bound(np.abs(a).T @ np.abs(d), batch)), f"layer {i} dW"
        assert np.all(np.abs(db - d.sum(axis=0)) <= accum_bound(np.abs(d).sum(axis=0), batch)), f"layer {i} db"
        assert np.any(db != 0)
    act1 = stored(net.activation_ptr(1), batch * cfg.layers[0].c_out).reshape(batch, -1)
    assert np.all(dz[0][act1 <= 0] == 0)
    assert mdnn.read_scaler(net.scaler)["good_steps"] == 1


@pytest.mark.timeout(300)
@pytest.mark.parametrize("case", ["lenet_bf16", "mlp784_fp32", "mlp_f16_scaled", "mlp_bf16_b1000"])
def test_classifier_head_from_stored_values(mdnn, case):
    """The classifier head of one step (cross-entropy over <= 32 classes: the
    loss kernel also sums the bias gradient from the dZ it stores), checked on
    the GPU's own stored logits, labels and layer input: dZ = S (softmax -
    onehot) / B rounded once to the storage type, the loss the batch mean of
    logsumexp - z[label], db = column sums of the stored dZ and dW = X^T dZ
    (bar gamma_B * sum |terms|, plus one storage step wherever fp32 softmax
    arithmetic may round dZ either way).  Cases: LeNet bf16 (batch 256), the
    fp32 MLP, an fp16 MLP with dynamic loss scaling (the bias sums carry the
    overflow test), and 1000 rows (most of the kernel's 1024 threads, ragged
    row segments)."""
    import dataclasses
    import torch
    from oracle.rounding import round_to
    from tests.helpers import accum_bound
    cfg = {"lenet_bf16": W.lenet_bf16(), "mlp784_fp32": W.mlp784_fp32(),
           "mlp_f16_scaled": dataclasses.replace(W.mlp784_fp32(), dtype="f16", loss_scaling=True,
                                                 init_scale=2.0 ** 10),
           "mlp_bf16_b1000": dataclasses.replace(W.mlp784_fp32(), dtype="bf16", batch=1000)}[case]
    net = _gpu_net(mdnn, cfg)
    x, t = W.batch_inputs(cfg, 0)
    loss = float(net.step(dev(x, "f32"), _target(cfg, t)).item())
    torch.cuda.synchronize()
    B, L = cfg.batch, len(cfg.layers)
    C, K = cfg.layers[-1].c_out, cfg.layers[-1].c_in
    es = 4 if cfg.dtype == "f32" else 2
    st = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[cfg.dtype]

    def stored(ptr, n, typ=st, size=es):
        off = ptr - net.ws.data_ptr()
        return net.ws[off:off + size * n].clone().view(typ).float().cpu().numpy().astype(np.float64)

    a = stored(net.activation_ptr(L - 1), B * K).reshape(B, K)
    z = stored(net.activation_ptr(L), B * C, torch.float32, 4).reshape(B, C)
    scale = cfg.init_scale if cfg.loss_scaling else 1.0
    zmax = z.max(axis=1, keepdims=True)
    lse = zmax[:, 0] + np.log(np.exp(z - zmax).sum(axis=1))
    p = np.exp(z - lse[:, None])
    onehot = np.zeros_like(p)
    onehot[np.arange(B), t] = 1.0
    want = scale * (p - onehot) / B
    # fp32 softmax arithmetic (exp, log, a product and a difference) before
    # the one rounding: a few fp32 ulps of the terms
    tol = 16 * 2.0 ** -24 * (np.abs(scale * p / B) + np.abs(want)) + 1e-38
    lo = round_to(want - tol, cfg.dtype) if cfg.dtype != "f32" else want - tol
    hi = round_to(want + tol, cfg.dtype) if cfg.dtype != "f32" else want + tol
    if L == 2:
        # the head's dZ buffer is not reused by a later layer: check it and use it
        d = stored(net.output_grad_ptr(0), B * C).reshape(B, C)
        assert np.all((d >= lo) & (d <= hi)), "dZ"
        slack = np.zeros_like(d)
    else:
        d = round_to(want, cfg.dtype)
        slack = hi - lo
    assert abs(loss - float(np.mean(lse - z[np.arange(B), t]))) <= 1e-5 * abs(loss)
    g = net.grads.cpu().numpy().astype(np.float64)
    wo, bo = cfg.param_offsets()[-1]
    db = g[bo:bo + C]
    dw = g[wo:wo + K * C].reshape(K, C)
    assert np.all(np.abs(db - d.sum(axis=0)) <= accum_bound(np.abs(d).sum(axis=0), B + 1) + slack.sum(axis=0)), "db"
    assert np.all(np.abs(dw - a.T @ d) <= accum_bound(np.abs(a).T @ np.abs(d), B + 1) + np.abs(a).T @ slack), "dW"
    assert np.any(db != 0)
    if cfg.loss_scaling:
        assert mdnn.read_scaler(net.scaler)["good_steps"] == 1
