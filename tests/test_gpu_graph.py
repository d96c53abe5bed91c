"""Recorded train steps (HIP graphs): a replay runs the same kernels in the
same order as mdnn_train_step, and every kernel of the synchronous step is
deterministic, so each replay must match an eager step on a twin net bit for
bit: loss, master weights, momentum and the loss scaler.  Replays alternate
with eager work of the program (other GEMMs, torch ops) and host
synchronisations, and cycle over several recorded batches.
"""
import dataclasses

import numpy as np
import pytest

import workloads as W
from tests.helpers import DT, dev

pytestmark = pytest.mark.gpu

CONFIGS = {
    "mlp_fp32": W.mlp784_fp32,
    "lenet_bf16": W.lenet_bf16,
    "wide_fp16_scaled": lambda: dataclasses.replace(W.wide_mlp_fp16(batch=256, width=512), lr=1e-4),
}


def _net(mdnn, cfg, params):
    net = mdnn.Net(cfg.layers, cfg.batch, DT[cfg.dtype], cfg.loss, cfg.lr, cfg.momentum,
                   cfg.loss_scaling, cfg.init_scale, cfg.n_classes)
    net.set_params(params)
    return net


def _target(cfg, t):
    return dev(t, "f32") if cfg.loss == W.LOSS_MSE else dev(t, "i32")


@pytest.mark.parametrize("name", list(CONFIGS))
def test_replays_match_eager_steps(mdnn, name):
    import torch
    cfg = CONFIGS[name]()
    params = W.init_params(cfg)
    eager, rec = _net(mdnn, cfg, params), _net(mdnn, cfg, params)
    batches = [W.batch_inputs(cfg, s) for s in range(3)]
    dev_b = [(dev(x, "f32"), _target(cfg, t)) for x, t in batches]
    losses = [torch.zeros(1, device="cuda") for _ in dev_b]
    graphs = [rec.record_step(x, t, loss_out=l) for (x, t), l in zip(dev_b, losses)]
    torch.cuda.synchronize()
    # recording runs nothing
    assert torch.equal(rec.master, eager.master)
    noise = torch.randn(300, 300, device="cuda", dtype=torch.float16)
    for i in range(7):
        x, t = dev_b[i % 3]
        le = float(eager.step(x, t).item())
        graphs[i % 3].launch()
        torch.cuda.synchronize()
        lr = float(losses[i % 3].item())
        assert lr == le, (i, lr, le)
        assert torch.equal(rec.master, eager.master), i
        if eager.mom is not None:
            assert torch.equal(rec.mom, eager.mom), i
        if eager.lowp is not None:
            assert torch.equal(rec.lowp, eager.lowp), i
        if eager.scaler is not None:
            assert mdnn.read_scaler(rec.scaler) == mdnn.read_scaler(eager.scaler), i
        # the program's own eager work between replays
        mdnn.gemm(mdnn.NN, noise, noise, out_dtype=torch.float32)
        (noise.float() @ noise.float()).sum().item()
    assert np.isfinite(le)
    for g in graphs:
        g.close()


def test_replay_on_another_stream_and_back_to_back(mdnn):
    """Replays queued back to back on a side stream equal the same number of
    eager steps."""
    import torch
    cfg = W.mlp784_fp32()
    params = W.init_params(cfg)
    eager, rec = _net(mdnn, cfg, params), _net(mdnn, cfg, params)
    x, t = W.batch_inputs(cfg, 5)
    X, T = dev(x, "f32"), _target(cfg, t)
    g = rec.record_step(X, T)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    for _ in range(5):
        g.launch(stream=s)
        eager.step(X, T)
    torch.cuda.synchronize()
    assert torch.equal(rec.master, eager.master)
    assert torch.equal(rec.loss, eager.loss)
    g.close()
