"""Pins of the oracle's per-operation definitions.

Each pin is independent of the oracle's own formula: pure-Python brute force on
tiny inputs, adjoint identities tying the backward ops to the forward op,
special cases that reduce to a plain matrix product or the identity, closed
forms (ln 10 for uniform logits over ten classes) and scipy's log_softmax.
"""
import itertools
import math

import numpy as np
import pytest

from oracle import ops


def _brute_gemm(layout, a, b, alpha, beta, c):
    if layout == "TN":
        k, m = a.shape
    else:
        m, k = a.shape
    n = b.shape[0] if layout == "NT" else b.shape[1]
    d = np.zeros((m, n))
    for i in range(m):
        for j in range(n):
            s = 0.0
            for p in range(k):
                av = a[p][i] if layout == "TN" else a[i][p]
                bv = b[j][p] if layout == "NT" else b[p][j]
                s += av * bv
            d[i][j] = alpha * s + (beta * c[i][j] if beta != 0 else 0.0)
    return d


@pytest.mark.parametrize("layout", ["NN", "NT", "TN"])
def test_gemm_brute_force(layout):
    g = np.random.default_rng(1)
    m, n, k = 5, 7, 6
    a = g.standard_normal((k, m) if layout == "TN" else (m, k))
    b = g.standard_normal((n, k) if layout == "NT" else (k, n))
    c = g.standard_normal((m, n))
    for alpha, beta in [(1.0, 0.0), (0.5, 1.0), (-2.0, 0.25)]:
        want = _brute_gemm(layout, a, b, alpha, beta, c)
        got = ops.gemm(layout, a, b, alpha, beta, c)
        assert np.allclose(got, want, rtol=1e-13, atol=1e-13)


def test_gemm_beta_zero_ignores_c():
    a = np.ones((2, 3))
    b = np.ones((3, 2))
    c = np.full((2, 2), np.nan)
    assert np.array_equal(ops.gemm("NN", a, b, 1.0, 0.0, c), np.full((2, 2), 3.0))


def test_gemm_forms_are_fc_layer_products():
    """NT of dY with W equals dY W^T; TN of X with dY equals X^T dY, and the
    adjoint <X W, G> = <X, G W^T> = <W, X^T G> ties the three forms together."""
    g = np.random.default_rng(2)
    x, w, gy = g.standard_normal((6, 4)), g.standard_normal((4, 3)), g.standard_normal((6, 3))
    y = ops.gemm("NN", x, w)
    dx = ops.gemm("NT", gy, w)          # B stored [N,K] = W[in,out] with N=in, K=out
    dw = ops.gemm("TN", x, gy)
    assert dx.shape == x.shape and dw.shape == w.shape
    ip = (y * gy).sum()
    assert abs(ip - (x * dx).sum()) < 1e-12 and abs(ip - (w * dw).sum()) < 1e-12


def test_gemm_integer_exact():
    g = np.random.default_rng(3)
    a = g.integers(-4, 5, (33, 100)).astype(np.float64)
    b = g.integers(-4, 5, (100, 17)).astype(np.float64)
    d = ops.gemm("NN", a, b)
    assert np.array_equal(d, np.rint(d))
    assert np.array_equal(d, _brute_gemm("NN", a, b, 1.0, 0.0, None))


# ---------------------------------------------------------------------------
# convolution
# ---------------------------------------------------------------------------

def _brute_conv(x, w, pad):
    n, h, wd, c = x.shape
    k, r, s, _ = w.shape
    ho, wo = h + 2 * pad - r + 1, wd + 2 * pad - s + 1
    y = np.zeros((n, ho, wo, k))
    for a, i, j, kk in itertools.product(range(n), range(ho), range(wo), range(k)):
        acc = 0.0
        for p, q, cc in itertools.product(range(r), range(s), range(c)):
            hh, ww = i + p - pad, j + q - pad
            if 0 <= hh < h and 0 <= ww < wd:
                acc += x[a, hh, ww, cc] * w[kk, p, q, cc]
        y[a, i, j, kk] = acc
    return y


@pytest.mark.parametrize("shape", [(2, 5, 4, 3, 2, 3, 3, 1), (1, 6, 6, 2, 3, 5, 5, 2),
                                   (2, 4, 5, 1, 2, 3, 3, 0), (1, 3, 3, 2, 2, 5, 5, 1)])
def test_conv_fwd_brute_force(shape):
    n, h, w, c, k, r, s, pad = shape
    g = np.random.default_rng(4)
    x = g.standard_normal((n, h, w, c))
    wt = g.standard_normal((k, r, s, c))
    assert np.allclose(ops.conv2d_fwd(x, wt, pad), _brute_conv(x, wt, pad), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("shape", [(2, 5, 4, 3, 2, 3, 3, 1), (1, 6, 6, 2, 3, 5, 5, 2),
                                   (2, 4, 5, 1, 2, 3, 3, 0), (1, 3, 3, 2, 2, 5, 5, 1)])
def test_conv_backward_adjoints(shape):
    """<conv(x,w), dy> = <x, bwd_data(dy,w)> = <w, bwd_filter(x,dy)>."""
    n, h, w, c, k, r, s, pad = shape
    g = np.random.default_rng(5)
    x = g.standard_normal((n, h, w, c))
    wt = g.standard_normal((k, r, s, c))
    y = ops.conv2d_fwd(x, wt, pad)
    dy = g.standard_normal(y.shape)
    dx = ops.conv2d_bwd_data(dy, wt, pad, h, w)
    dw = ops.conv2d_bwd_filter(x, dy, pad, r, s)
    ip = (y * dy).sum()
    assert abs(ip - (x * dx).sum()) <= 1e-12 * max(1.0, abs(ip))
    assert abs(ip - (wt * dw).sum()) <= 1e-12 * max(1.0, abs(ip))
    # and each backward op against a brute-force derivative of the forward
    # (linearity: the gradient of <conv(x,w),dy> w.r.t. x[e] is conv(e,w)·dy)
    e = np.zeros_like(x)
    e[0, h // 2, w // 2, c - 1] = 1.0
    assert abs((_brute_conv(e, wt, pad) * dy).sum() - dx[0, h // 2, w // 2, c - 1]) < 1e-12
    e = np.zeros_like(wt)
    e[k - 1, r // 2, 0, 0] = 1.0
    assert abs((_brute_conv(x, e, pad) * dy).sum() - dw[k - 1, r // 2, 0, 0]) < 1e-12


def test_conv_1x1_is_gemm():
    g = np.random.default_rng(6)
    x = g.standard_normal((2, 3, 4, 5))
    w = g.standard_normal((6, 1, 1, 5))
    y = ops.conv2d_fwd(x, w, 0)
    assert np.allclose(y.reshape(-1, 6), x.reshape(-1, 5) @ w[:, 0, 0, :].T, rtol=1e-13, atol=1e-13)


def test_conv_delta_filter_is_identity():
    g = np.random.default_rng(7)
    x = g.standard_normal((2, 5, 5, 3))
    w = np.zeros((3, 3, 3, 3))
    for cc in range(3):
        w[cc, 1, 1, cc] = 1.0
    assert np.array_equal(ops.conv2d_fwd(x, w, 1), x)
    # shifted delta moves the image by one pixel (zero padding enters)
    w2 = np.zeros((3, 3, 3, 3))
    for cc in range(3):
        w2[cc, 2, 1, cc] = 1.0          # reads x[h+1]
    y = ops.conv2d_fwd(x, w2, 1)
    assert np.array_equal(y[:, :-1], x[:, 1:]) and np.all(y[:, -1] == 0)


# ---------------------------------------------------------------------------
# bias / relu / maxpool
# ---------------------------------------------------------------------------

def test_bias_relu_brute_force():
    g = np.random.default_rng(8)
    x = g.standard_normal((5, 4))
    b = g.standard_normal(4)
    y = ops.bias_act(x, b, "relu")
    for i, j in itertools.product(range(5), range(4)):
        v = x[i, j] + b[j]
        assert y[i, j] == (v if v > 0 else 0.0)
    dy = g.standard_normal((5, 4))
    dz, db = ops.bias_act_bwd(dy, y, "relu")
    for j in range(4):
        s = 0.0
        for i in range(5):
            s += dy[i, j] if y[i, j] > 0 else 0.0
        assert abs(db[j] - s) < 1e-14
    assert np.all(ops.relu(np.array([np.nan])) != 0)   # NaN propagates
    assert ops.relu_mask(np.array([0.0, -0.0, 1e-30]))[:2].sum() == 0


def test_maxpool_brute_force_with_ties():
    g = np.random.default_rng(9)
    x = g.integers(0, 3, (2, 6, 8, 3)).astype(np.float64)   # many ties
    y, arg = ops.maxpool2_fwd(x)
    n, h, w, c = x.shape
    for a, i, j, cc in itertools.product(range(n), range(h // 2), range(w // 2), range(c)):
        win = [x[a, 2 * i + di, 2 * j + dj, cc] for di in (0, 1) for dj in (0, 1)]
        best = 0
        for t in range(1, 4):
            if win[t] > win[best]:
                best = t
        assert y[a, i, j, cc] == win[best] and arg[a, i, j, cc] == best
    dy = g.standard_normal(y.shape)
    dx = ops.maxpool2_bwd(dy, arg, h, w)
    for a, i, j, cc in itertools.product(range(n), range(h // 2), range(w // 2), range(c)):
        di, dj = divmod(int(arg[a, i, j, cc]), 2)
        blk = dx[a, 2 * i:2 * i + 2, 2 * j:2 * j + 2, cc]
        assert blk[di, dj] == dy[a, i, j, cc] and np.count_nonzero(blk) <= 1
    # adjoint: <pool(x) selection, dy> = <x, bwd(dy)>
    assert abs((y * dy).sum() - (x * dx).sum()) < 1e-12


# ---------------------------------------------------------------------------
# losses
# ---------------------------------------------------------------------------

def test_softmax_uniform_logits_ln10():
    b = 16
    labels = np.arange(b) % 10
    loss, dz = ops.softmax_xent(np.zeros((b, 10)), labels)
    assert loss == pytest.approx(2.302585092994046, abs=1e-15)
    assert loss == pytest.approx(math.log(10.0), abs=1e-15)
    onehot = np.eye(10)[labels]
    assert np.allclose(dz, (0.1 - onehot) / b, atol=1e-17)


def test_softmax_invariants_and_library():
    scipy_special = pytest.importorskip("scipy.special")
    g = np.random.default_rng(10)
    z = g.standard_normal((32, 10)) * 4
    lab = g.integers(0, 10, 32)
    loss, dz = ops.softmax_xent(z, lab, scale=8.0)
    p = dz * 32 / 8.0 + np.eye(10)[lab]          # recover softmax
    assert np.allclose(p.sum(axis=1), 1.0, atol=1e-14)
    assert np.allclose(dz.sum(axis=1), 0.0, atol=1e-14)
    ls = scipy_special.log_softmax(z, axis=1)
    assert loss == pytest.approx(-ls[np.arange(32), lab].mean(), rel=1e-14)
    assert np.allclose(p, np.exp(ls), atol=1e-14)
    loss2, dz2 = ops.softmax_xent(z + 1000.0, lab, scale=8.0)
    assert loss2 == pytest.approx(loss, rel=1e-12) and np.allclose(dz2, dz, atol=1e-13)


def test_softmax_bad_label_is_nan():
    loss, dz = ops.softmax_xent(np.zeros((3, 10)), np.array([0, 10, -1]))
    assert math.isnan(loss) and np.all(np.isnan(dz[1:])) and np.all(np.isfinite(dz[0]))


def test_mse_closed_forms():
    g = np.random.default_rng(11)
    t = g.standard_normal((64, 1))
    loss, dy = ops.mse_loss(np.zeros((64, 1)), t)
    assert loss == pytest.approx(float((t ** 2).mean()), rel=1e-14)
    assert np.allclose(dy, -2 * t / 64)
    y = g.standard_normal((64, 1))
    loss, dy = ops.mse_loss(y, t, scale=4.0)
    assert loss == pytest.approx(sum((y[i, 0] - t[i, 0]) ** 2 for i in range(64)) / 64, rel=1e-13)
    assert np.allclose(dy, 4.0 * 2 * (y - t) / 64)


# ---------------------------------------------------------------------------
# SGD / momentum / loss scaler
# ---------------------------------------------------------------------------

def test_sgd_quadratic_closed_form():
    """f = 0.5 |w|^2 has gradient w, so plain SGD gives w_{t+1} = (1 - lr) w_t."""
    w0 = np.array([1.0, -2.0, 3.0])
    w = w0.copy()
    for t in range(1, 6):
        w, _, _, ok = ops.sgd_update(w, w, None, 0.1, 0.0, None)
        assert ok and np.allclose(w, 0.9 ** t * w0, rtol=1e-14)


def test_momentum_constant_gradient_closed_form():
    g = np.array([0.5, -1.0])
    w, v = np.zeros(2), np.zeros(2)
    mu, lr = 0.9, 0.01
    wsum = np.zeros(2)
    for t in range(1, 8):
        w, v, _, _ = ops.sgd_update(w, g, v, lr, mu, None)
        vt = g * (1 - mu ** t) / (1 - mu)
        wsum += vt
        assert np.allclose(v, vt, rtol=1e-13) and np.allclose(w, -lr * wsum, rtol=1e-13)


def test_scaler_overflow_skips_and_halves():
    sc = ops.new_scaler(2.0 ** 16)
    w, v = np.ones(4), np.full(4, 0.25)
    g = np.array([1.0, np.inf, 0.0, 1.0])
    w2, v2, sc2, ok = ops.sgd_update(w, g, v, 0.1, 0.9, sc)
    assert not ok and np.array_equal(w2, w) and np.array_equal(v2, v)
    assert sc2["scale"] == 2.0 ** 15 and sc2["good_steps"] == 0 and sc2["overflow"] == 1
    g = np.array([1.0, np.nan, 0.0, 1.0])
    _, _, sc3, ok = ops.sgd_update(w, g, v, 0.1, 0.9, ops.new_scaler(1.0))
    assert not ok and sc3["scale"] == 1.0            # never below min_scale


def test_scaler_unscales_and_grows():
    sc = ops.new_scaler(8.0, growth_interval=3)
    w = np.zeros(2)
    for t in range(3):
        w, _, sc, ok = ops.sgd_update(w, np.array([8.0, -16.0]), None, 1.0, 0.0, sc)
        assert ok
    assert np.array_equal(w, np.array([-3.0, 6.0]))   # g/S = (1,-2) three times
    assert sc["scale"] == 16.0 and sc["good_steps"] == 0
