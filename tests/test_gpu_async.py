"""Asynchronous SGD on one GPU (section 3.1): workers on separate streams
share one fp32 parameter vector and add their updates to it with atomics.

The execution is non-deterministic by design, so parity is:
* exact where the outcome does not depend on the interleaving: concurrent
  update calls of known steps lose nothing (the final weights are exact), and
  one worker is plain SGD (loss trajectory within 1e-3 of the oracle's);
* statistical against the oracle's bounded-staleness model otherwise: after
  120 updates by four workers the held-out loss is within 5% of the model's
  (staleness 3), both well below the starting loss (the synthetic labels are
  random, so training calibrates the outputs towards ln 10);
* low-precision workers (per-worker snapshots of the shared weights) lower
  their loss, and loss-scaled workers (per-worker scalers) stay finite and
  within a factor 2 of the model's losses.
"""
import dataclasses
import numpy as np
import pytest

import workloads as W
from oracle import async_sgd, train
from tests.helpers import DT, dev

pytestmark = pytest.mark.gpu


def _target(cfg, t):
    return dev(t, "f32") if cfg.loss == W.LOSS_MSE else dev(t, "i32")


def _workers(mdnn, cfg, n, params):
    first = mdnn.Net(cfg.layers, cfg.batch, DT[cfg.dtype], cfg.loss, cfg.lr, cfg.momentum,
                     cfg.loss_scaling, cfg.init_scale, cfg.n_classes)
    first.set_params(params)
    nets = [first]
    for _ in range(n - 1):
        w = mdnn.Net(cfg.layers, cfg.batch, DT[cfg.dtype], cfg.loss, cfg.lr, cfg.momentum,
                     cfg.loss_scaling, cfg.init_scale, cfg.n_classes, shared_master=first.master)
        nets.append(w)
    return nets


def test_concurrent_updates_lose_nothing(mdnn):
    import torch
    n, workers, reps, lr = 1 << 20, 4, 25, 0.5
    w = torch.full((n,), 1024.0, dtype=torch.float32, device="cuda")
    g = torch.ones(n, dtype=torch.float32, device="cuda")
    streams = [torch.cuda.Stream() for _ in range(workers)]
    torch.cuda.synchronize()
    for _ in range(reps):
        for s in streams:
            mdnn.mdnn_sgd_update_async(n, w, g, None, lr, 0.0, None, stream=s)
    torch.cuda.synchronize()
    # every step is a multiple of 0.5 on values >= 974: all sums are exact
    assert torch.all(w == 1024.0 - lr * workers * reps)


def test_async_update_matches_sync_update_alone(mdnn):
    """One caller: the atomic update is w + (-lr*v), the plain one
    fma(-lr, v, w); they differ by at most one rounding of the operands,
    momentum and loss scaling included."""
    import torch
    n = 100003
    g0 = torch.randn(n, device="cuda") * 64
    w_a = torch.randn(n, device="cuda")
    w_b = w_a.clone()
    v_a = torch.randn(n, device="cuda")
    v_b = v_a.clone()
    sa, sb = mdnn.make_scaler(64.0), mdnn.make_scaler(64.0)
    mdnn.mdnn_sgd_update_async(n, w_a, g0, v_a, 0.01, 0.9, sa)
    mdnn.mdnn_sgd_update(n, w_b, g0, v_b, None, mdnn.F32, 0.01, 0.9, sb)
    torch.cuda.synchronize()
    assert torch.equal(v_a, v_b)
    # the atomic path rounds -lr*v before the add: one rounding of each
    # operand's size, which dominates where w and lr*v nearly cancel
    bound = (torch.abs(w_b) + 0.01 * torch.abs(v_a)) * 2.0 ** -23
    assert torch.all(torch.abs(w_a - w_b) <= bound)
    assert mdnn.read_scaler(sa) == mdnn.read_scaler(sb)


def test_single_worker_is_plain_sgd(mdnn):
    import torch
    cfg = W.mlp784_fp32()
    params = W.init_params(cfg)
    net = _workers(mdnn, cfg, 1, params)[0]
    batches = [W.batch_inputs(cfg, s) for s in range(10)]
    gl = [float(net.step_async(dev(x, "f32"), _target(cfg, t)).item()) for x, t in batches]
    ol = async_sgd.async_train(train.from_config(cfg, params), batches, workers=1)
    for s, (a, b) in enumerate(zip(gl, ol)):
        assert abs(a - b) <= 1e-3 * abs(b), (s, gl, ol)
    del torch


def test_four_workers_track_the_staleness_model(mdnn):
    import torch
    cfg = W.mlp784_fp32()
    params = W.init_params(cfg)
    workers, rounds = 4, 30
    nets = _workers(mdnn, cfg, workers, params)
    streams = [torch.cuda.Stream() for _ in range(workers)]
    batches = [W.batch_inputs(cfg, s) for s in range(workers * rounds)]
    dev_b = [(dev(x, "f32"), _target(cfg, t)) for x, t in batches]
    torch.cuda.synchronize()
    for r in range(rounds):
        for k in range(workers):
            x, t = dev_b[r * workers + k]
            nets[k].step_async(x, t, stream=streams[k])
    torch.cuda.synchronize()
    w_gpu = nets[0].master.cpu().numpy().astype(np.float64)
    model = train.from_config(cfg, params)
    async_sgd.async_train(model, batches, workers=workers)
    xe, te = W.batch_inputs(cfg, 10 ** 4)               # held-out batch
    start = train.from_config(cfg, params).loss_only(xe, te)
    gpu_eval = train.from_config(cfg, w_gpu).loss_only(xe, te)
    model_eval = model.loss_only(xe, te)
    assert gpu_eval < 0.9 * start and model_eval < 0.9 * start, (start, gpu_eval, model_eval)
    assert abs(gpu_eval - model_eval) <= 0.05 * model_eval, (gpu_eval, model_eval)


def _two_workers(mdnn, cfg, steps):
    import torch
    params = W.init_params(cfg)
    nets = _workers(mdnn, cfg, 2, params)
    streams = [torch.cuda.Stream() for _ in range(2)]
    losses = [torch.zeros(1, device="cuda") for _ in range(steps)]
    batches = [W.batch_inputs(cfg, s) for s in range(steps)]
    torch.cuda.synchronize()
    for i, (x, t) in enumerate(batches):
        nets[i % 2].step_async(dev(x, "f32"), _target(cfg, t), loss_out=losses[i], stream=streams[i % 2])
    torch.cuda.synchronize()
    model = async_sgd.async_train(train.from_config(cfg, params), batches, workers=2)
    return [float(l.item()) for l in losses], model, nets


def test_lowp_workers_train(mdnn):
    ls, model, _ = _two_workers(mdnn, W.lenet_bf16(), 16)
    assert all(np.isfinite(ls))
    assert np.mean(ls[-4:]) < 0.95 * np.mean(ls[:4]), ls
    assert np.mean(model[-4:]) < 0.95 * np.mean(model[:4])


def test_loss_scaled_workers(mdnn):
    cfg = dataclasses.replace(W.wide_mlp_fp16(batch=512, width=1024), lr=1e-4)
    ls, model, nets = _two_workers(mdnn, cfg, 16)
    assert all(np.isfinite(ls))
    g, m = np.mean(ls[-8:]), np.mean(model[-8:])
    assert 0.5 * m <= g <= 2.0 * m, (ls, model)
    for n in nets:
        sc = mdnn.read_scaler(n.scaler)
        assert sc["scale"] >= 1.0 and sc["reserved"] == 0
