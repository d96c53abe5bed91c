"""GPU parity of the memory-bound kernels against the oracle: precision
conversion (bit-exact RNE), bias+ReLU forward/backward, 2x2 max pooling
(bit-exact, ties included), softmax cross-entropy, MSE and the SGD / momentum
update with dynamic loss scaling."""
import math

import numpy as np
import pytest

import workloads as W
from oracle import ops
from oracle.rounding import decode, round_to
from tests.helpers import DT, dev, empty, host64, lowp_close, norm_max_err

pytestmark = pytest.mark.gpu


def _special_f32():
    """fp32 values around every fp16 / bf16 rounding boundary, subnormals,
    overflow thresholds, infinities and NaN."""
    g = np.random.default_rng(21)
    parts = [g.standard_normal(200_000).astype(np.float32),
             (g.standard_normal(100_000) * np.exp2(g.integers(-30, 20, 100_000))).astype(np.float32),
             np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 65504.0, 65519.996, 65520.0, 1e38,
                       3.3e38, -3.4e38, 2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -25, 1e-40], np.float32)]
    h = np.arange(0, 65536, 7, dtype=np.uint32).astype(np.uint16).view(np.float16).astype(np.float64)
    h = np.unique(h[np.isfinite(h)])
    mids = ((h[:-1] + h[1:]) / 2).astype(np.float32)
    parts += [mids, np.nextafter(mids, np.float32(np.inf)), np.nextafter(mids, np.float32(-np.inf))]
    b = (np.arange(0, 65536, 5, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)
    b = np.unique(b[np.isfinite(b)])
    bm = ((b[:-1] + b[1:]) / 2).astype(np.float32)
    parts += [bm, np.nextafter(bm, np.float32(np.inf)), np.nextafter(bm, np.float32(-np.inf))]
    return np.concatenate(parts)


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_cast_round_to_nearest_even_bitexact(mdnn, dt):
    import torch
    x = _special_f32()
    src = dev(x, "f32")
    dst = empty(x.shape, dt)
    mdnn.mdnn_cast(x.size, src, DT["f32"], dst, DT[dt])
    back = empty(x.shape, "f32")
    mdnn.mdnn_cast(x.size, dst, DT[dt], back, DT["f32"])
    torch.cuda.synchronize()
    got = host64(dst)
    with np.errstate(over="ignore"):
        want = round_to(x.astype(np.float64), dt)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])
    assert np.array_equal(host64(back)[~nan], want[~nan])          # widening is exact
    # odd length and unaligned start take the element-wise path
    mdnn.mdnn_cast(1001, src[3:], DT["f32"], dst[1:], DT[dt])
    torch.cuda.synchronize()
    assert np.array_equal(host64(dst)[1:1002][~nan[3:1004]], want[3:1004][~nan[3:1004]])


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_bias_act_fwd_bwd(mdnn, dt):
    import torch
    rows, cols = 300, 77
    x = W.normal((rows, cols), 22, 1, "f32")
    b = W.normal((cols,), 22, 2, "f32")
    y = empty((rows, cols), dt)
    mdnn.mdnn_bias_act_fwd(rows, cols, dev(x, "f32"), dev(b, "f32"), mdnn.ACT_RELU, y, DT[dt])
    dy = W.normal((rows, cols), 22, 3, dt)
    dz = empty((rows, cols), dt)
    db = torch.empty(cols, dtype=torch.float32, device="cuda")
    mdnn.mdnn_bias_act_bwd(rows, cols, dev(dy, dt), y, mdnn.ACT_RELU, dz, db, DT[dt])
    db2 = torch.empty(cols, dtype=torch.float32, device="cuda")
    nws = mdnn.mdnn_bias_act_bwd_workspace(rows, cols)
    ws = torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda")
    mdnn.mdnn_bias_act_bwd(rows, cols, dev(dy, dt), y, mdnn.ACT_RELU, None, db2, DT[dt], ws, nws)
    torch.cuda.synchronize()
    exact = ops.bias_act(x.astype(np.float64), b.astype(np.float64), "relu")
    # x + b is rounded to fp32 before the storage rounding
    assert lowp_close(host64(y), exact, dt, 2.0 ** -24 * np.abs(exact))
    if dt == "f32":
        assert np.array_equal(host64(y), round_to(exact, "f32"))
    dzw, dbw = ops.bias_act_bwd(decode(dy, dt), host64(y), "relu")
    assert np.array_equal(host64(dz), dzw)
    assert norm_max_err(host64(db), dbw) <= 1e-5
    assert norm_max_err(host64(db2), dbw) <= 1e-5      # two-pass reduction with a workspace


@pytest.mark.parametrize("shape", [(200704, 32), (4096, 4096), (1000, 10), (513, 72)])
def test_column_sums_tall_and_wide(mdnn, shape):
    """Bias gradients of the workloads' layer shapes (conv1 of the LeNet-style
    net: 200704 x 32; a wide FC layer: 4096 x 4096), two-pass, deterministic."""
    import torch
    rows, cols = shape
    dy = W.normal((rows, cols), 29, 1, "f16", 0.01)
    DY = dev(dy, "f16")
    nws = mdnn.mdnn_bias_act_bwd_workspace(rows, cols)
    ws = torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda")
    db = torch.empty(cols, dtype=torch.float32, device="cuda")
    db2 = torch.empty(cols, dtype=torch.float32, device="cuda")
    mdnn.mdnn_bias_act_bwd(rows, cols, DY, None, mdnn.ACT_NONE, None, db, DT["f16"], ws, nws)
    mdnn.mdnn_bias_act_bwd(rows, cols, DY, None, mdnn.ACT_NONE, None, db2, DT["f16"], ws, nws)
    torch.cuda.synchronize()
    assert norm_max_err(host64(db), dy.astype(np.float64).sum(axis=0)) <= 1e-5
    assert torch.equal(db, db2)


@pytest.mark.parametrize("shape,dt", [((256, 1024), "bf16"), ((37, 72), "f16"), ((200, 77), "f32"), ((1, 8), "bf16"),
                                      ((256, 10), "f16")])
def test_column_sums_short(mdnn, shape, dt):
    """At most 256 rows (a classifier's hidden layer at batch 256): one pass,
    masked by a ReLU output and unmasked, against the exact sums."""
    import torch
    rows, cols = shape
    dy = W.normal((rows, cols), 31, 1, dt)
    yv = W.normal((rows, cols), 31, 2, dt)
    DY, Y = dev(dy, dt), dev(yv, dt)
    db = torch.empty(cols, dtype=torch.float32, device="cuda")
    dbm = torch.empty(cols, dtype=torch.float32, device="cuda")
    dbm2 = torch.empty(cols, dtype=torch.float32, device="cuda")
    mdnn.mdnn_bias_act_bwd(rows, cols, DY, None, mdnn.ACT_NONE, None, db, DT[dt])
    mdnn.mdnn_bias_act_bwd(rows, cols, DY, Y, mdnn.ACT_RELU, None, dbm, DT[dt])
    mdnn.mdnn_bias_act_bwd(rows, cols, DY, Y, mdnn.ACT_RELU, None, dbm2, DT[dt])
    torch.cuda.synchronize()
    d64, y64 = decode(dy, dt), decode(yv, dt)
    assert norm_max_err(host64(db), d64.sum(axis=0)) <= 1e-5
    assert norm_max_err(host64(dbm), np.where(y64 > 0, d64, 0.0).sum(axis=0)) <= 1e-5
    assert torch.equal(dbm, dbm2)


# c = 12: element-wise kernels; c = 16 and 64 (16-bit types): eight channels
# per thread with 16-byte accesses
@pytest.mark.parametrize("c", [12, 16, 64])
@pytest.mark.parametrize("dt", ["f16", "bf16", "f32"])
def test_maxpool_bitexact_with_ties(mdnn, dt, c):
    import torch
    n, h, w = 3, 10, 14
    x = W.small_ints((n, h, w, c), 23, 1, lo=-2, hi=2, dtype=dt)     # many ties
    X = dev(x, dt)
    y = empty((n, h // 2, w // 2, c), dt)
    arg = torch.empty((n, h // 2, w // 2, c), dtype=torch.uint8, device="cuda")
    mdnn.mdnn_maxpool2_fwd(n, h, w, c, X, y, arg, DT[dt])
    dy = W.normal((n, h // 2, w // 2, c), 23, 2, dt)
    dx = empty((n, h, w, c), dt)
    dx.fill_(float("nan"))
    mdnn.mdnn_maxpool2_bwd(n, h, w, c, dev(dy, dt), arg, dx, DT[dt])
    torch.cuda.synchronize()
    yw, aw = ops.maxpool2_fwd(decode(x, dt))
    assert np.array_equal(host64(y), yw)
    assert np.array_equal(arg.cpu().numpy(), aw)
    assert np.array_equal(host64(dx), ops.maxpool2_bwd(decode(dy, dt), aw, h, w))


def test_maxpool_odd_sizes(mdnn):
    import torch
    n, h, w, c = 2, 7, 5, 3
    x = W.normal((n, h, w, c), 24, 1, "f16")
    X = dev(x, "f16")
    y = empty((n, 3, 2, c), "f16")
    arg = torch.empty((n, 3, 2, c), dtype=torch.uint8, device="cuda")
    mdnn.mdnn_maxpool2_fwd(n, h, w, c, X, y, arg, DT["f16"])
    dx = empty((n, h, w, c), "f16")
    mdnn.mdnn_maxpool2_bwd(n, h, w, c, y, arg, dx, DT["f16"])
    torch.cuda.synchronize()
    yw, aw = ops.maxpool2_fwd(decode(x, "f16"))
    assert np.array_equal(host64(y), yw)
    assert np.array_equal(host64(dx), ops.maxpool2_bwd(yw, aw, h, w))


# (256, 10) and (3000, 7): a thread per row (few classes; B > 1024 walks
# rows in turns); (100, 33) and (5, 1000): a wave per row.
@pytest.mark.parametrize("shape", [(256, 10), (3000, 7), (100, 33), (5, 1000)])
@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_softmax_xent(mdnn, dt, shape):
    import torch
    B, Cn = shape
    z = W.normal((B, Cn), 25, 1, "f32", 3.0)
    lab = W.rng(25, 2).integers(0, Cn, B).astype(np.int32)
    scale = torch.tensor([256.0], dtype=torch.float32, device="cuda")
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    dz = empty((B, Cn), dt)
    mdnn.mdnn_softmax_xent(B, Cn, dev(z, "f32"), Cn, dev(lab, "i32"), scale, loss, dz, Cn, DT[dt])
    torch.cuda.synchronize()
    lw, dzw = ops.softmax_xent(z.astype(np.float64), lab, 256.0)
    assert abs(loss.item() - lw) <= 1e-5 * abs(lw)
    assert norm_max_err(host64(dz), dzw) <= (1e-6 if dt == "f32" else 2.0 ** -8)


def test_softmax_uniform_logits_ln10_and_bad_labels(mdnn):
    import torch
    B = 64
    z = torch.zeros((B, 10), dtype=torch.float32, device="cuda")
    lab = torch.arange(B, dtype=torch.int32, device="cuda") % 10
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    dz = torch.empty((B, 10), dtype=torch.float32, device="cuda")
    mdnn.mdnn_softmax_xent(B, 10, z, 10, lab, None, loss, dz, 10, DT["f32"])
    torch.cuda.synchronize()
    assert loss.item() == pytest.approx(math.log(10.0), rel=2e-7)
    onehot = np.eye(10)[np.arange(B) % 10]
    assert np.allclose(dz.cpu().numpy(), (0.1 - onehot) / B, atol=1e-9)
    lab[3] = 10
    mdnn.mdnn_softmax_xent(B, 10, z, 10, lab, None, loss, dz, 10, DT["f32"])
    torch.cuda.synchronize()
    assert math.isnan(loss.item()) and torch.isnan(dz[3]).all() and torch.isfinite(dz[4]).all()


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_mse(mdnn, dt):
    import torch
    B = 4096
    y = W.normal((B, 1), 26, 1, "f32")
    t = W.normal((B, 1), 26, 2, "f32")
    scale = torch.tensor([65536.0], dtype=torch.float32, device="cuda")
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    dy = empty((B, 1), dt)
    mdnn.mdnn_mse_loss(B, 1, dev(y, "f32"), dev(t, "f32"), scale, loss, dy, DT[dt])
    torch.cuda.synchronize()
    lw, dyw = ops.mse_loss(y.astype(np.float64), t.astype(np.float64), 65536.0)
    assert abs(loss.item() - lw) <= 1e-5 * lw
    # y - t is rounded to fp32 before the storage rounding: allow that error
    assert lowp_close(host64(dy), dyw, dt, 2.0 ** -23 * np.abs(dyw))


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("momentum", [0.0, 0.9])
def test_sgd_update_against_oracle(mdnn, dt, momentum):
    import torch
    n = 100_003
    w = W.normal((n,), 27, 1, "f32")
    g = W.normal((n,), 27, 2, "f32", 1000.0)
    v = W.normal((n,), 27, 3, "f32", 0.1)
    wt, gt, vt = dev(w, "f32"), dev(g, "f32"), dev(v, "f32")
    wlp = empty((n,), dt)
    sc = mdnn.make_scaler(1024.0)
    mdnn.mdnn_sgd_update(n, wt, gt, vt if momentum else None, wlp, DT[dt], 0.01, momentum, sc)
    torch.cuda.synchronize()
    ww, vw, scw, ok = ops.sgd_update(w.astype(np.float64), g.astype(np.float64),
                                     v.astype(np.float64) if momentum else None, 0.01, momentum,
                                     ops.new_scaler(1024.0))
    assert ok
    assert np.max(np.abs(host64(wt) - ww)) <= 2.0 ** -23 * np.max(np.abs(ww)) * 2
    if momentum:
        assert np.max(np.abs(host64(vt) - vw)) <= 2.0 ** -23 * np.max(np.abs(vw)) * 2
    assert np.array_equal(host64(wlp), round_to(host64(wt), dt))
    s = mdnn.read_scaler(sc)
    assert s["scale"] == 1024.0 and s["good_steps"] == 1 and s["overflow"] == 0 and s["reserved"] == 0


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_sgd_vector_and_element_paths_agree(mdnn, dt):
    """16-byte aligned buffers take four parameters per thread (and the n % 4
    tail), an unaligned momentum buffer the element-wise kernel: same bits."""
    import torch
    n = 4099
    w = W.normal((n,), 28, 1, "f32")
    g = W.normal((n,), 28, 2, "f32")
    v = W.normal((n,), 28, 3, "f32")
    outs = []
    for off in (0, 1):
        wt, gt = dev(w, "f32"), dev(g, "f32")
        vbuf = torch.zeros(n + 1, dtype=torch.float32, device="cuda")
        vt = vbuf[off:off + n]
        vt.copy_(dev(v, "f32"))
        wlp = empty((n,), dt)
        mdnn.mdnn_sgd_update(n, wt, gt, vt, wlp, DT[dt], 0.05, 0.9, mdnn.make_scaler(8.0))
        torch.cuda.synchronize()
        outs.append((wt.clone(), vt.clone(), wlp.clone()))
    for a, b in zip(*outs):
        assert torch.equal(a, b)


def test_sgd_overflow_skips_and_halves(mdnn):
    import torch
    n = 4099
    w = W.normal((n,), 28, 1, "f32")
    g = W.normal((n,), 28, 2, "f32")
    g[1234] = np.inf
    wt, gt = dev(w, "f32"), dev(g, "f32")
    vt = torch.full((n,), 0.5, dtype=torch.float32, device="cuda")
    wlp = empty((n,), "f16")
    wlp.fill_(7.0)
    sc = mdnn.make_scaler(65536.0)
    mdnn.mdnn_sgd_update(n, wt, gt, vt, wlp, DT["f16"], 0.1, 0.9, sc)
    torch.cuda.synchronize()
    assert np.array_equal(host64(wt), w.astype(np.float64))
    assert torch.all(vt == 0.5) and torch.all(wlp == 7.0)
    s = mdnn.read_scaler(sc)
    assert s["scale"] == 32768.0 and s["overflow"] == 1 and s["good_steps"] == 0 and s["reserved"] == 0
    # NaN in the tail (not a multiple of 4) is caught too; scale never below min_scale
    g[1234] = 0.0
    g[n - 1] = np.nan
    sc1 = mdnn.make_scaler(1.0)
    mdnn.mdnn_sgd_update(n, wt, dev(g, "f32"), vt, wlp, DT["f16"], 0.1, 0.9, sc1)
    torch.cuda.synchronize()
    s = mdnn.read_scaler(sc1)
    assert s["scale"] == 1.0 and s["overflow"] == 1


def test_scaler_growth_after_interval(mdnn):
    import torch
    n = 64
    wt = torch.zeros(n, dtype=torch.float32, device="cuda")
    gt = torch.full((n,), 8.0, dtype=torch.float32, device="cuda")
    sc = mdnn.make_scaler(8.0, growth_interval=3)
    for _ in range(3):
        mdnn.mdnn_sgd_update(n, wt, gt, None, None, DT["f32"], 1.0, 0.0, sc)
    torch.cuda.synchronize()
    assert torch.all(wt == -3.0)
    s = mdnn.read_scaler(sc)
    assert s["scale"] == 16.0 and s["good_steps"] == 0
