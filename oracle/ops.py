"""fp64 definitions of every operation of one SGD step (test infrastructure only).

Every function takes and returns float64 arrays holding exact values; storage
rounding is the caller's business (``rounding.round_to``).  Layout conventions
(row-major everywhere):

* activations [B, F]; images NHWC [N, H, W, C];
* fully connected weights W[in, out], so the forward product is X @ W;
* convolution filters [Cout, R, S, Cin]; stride 1, zero padding ``pad``.
"""
from __future__ import annotations

from typing import Optional, Tuple

import numpy as np

NN, NT, TN = "NN", "NT", "TN"


# ---------------------------------------------------------------------------
# Dense contraction: section 3.2, the mixed-precision multiply-accumulate
# D = C + A*B (A, B low precision; C, D fp32).  Generalised with scalars to
# D = alpha * op(A) op(B) + beta * C; beta == 0 never reads C.
# ---------------------------------------------------------------------------

def gemm(layout: str, a: np.ndarray, b: np.ndarray, alpha: float = 1.0,
         beta: float = 0.0, c: Optional[np.ndarray] = None) -> np.ndarray:
    """NN: A[M,K] B[K,N]; NT: A[M,K] B[N,K] (B used transposed);
    TN: A[K,M] (used transposed) B[K,N].  These are a fully connected layer's
    forward (X W), backward-data (dY W^T) and backward-weight (X^T dY) forms."""
    op_a = a.T if layout == TN else a
    op_b = b.T if layout == NT else b
    d = alpha * (op_a @ op_b)
    if beta != 0.0:
        d = d + beta * c
    return d


# ---------------------------------------------------------------------------
# fp32 products from fp16 matrix-core products: section 3.2's Eq. (1).  An
# fp32 matrix is the scaled sum of two fp16 matrices, X ~ s1*X1 + s2*X2 with
# s2 = 2^-11 * s1 (the well-scaled case the section spells out, for a
# caller-chosen power of two s1): X1 = RNE16(X / s1) keeps the leading 11
# significant bits, X2 = RNE16((X - s1*X1) / s2) the next 11.  The product
# of two such matrices keeps three of the four fp16 products (the X2*Y2
# term, 2^-22 below the leading one, is dropped).
# ---------------------------------------------------------------------------

SPLIT_SHIFT = 2.0 ** -11   # s2 / s1


def split_f16(x: np.ndarray, scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """(X1, X2) of Eq. (1) as exact fp64 values of fp16 numbers."""
    from .rounding import round_to
    x = np.asarray(x, dtype=np.float64)
    hi = round_to(x / scale, "f16")
    with np.errstate(invalid="ignore"):
        lo = round_to((x - scale * hi) / (scale * SPLIT_SHIFT), "f16")
    return hi, lo


def split_scale(x: np.ndarray) -> float:
    """The leading scale s1 of Eq. (1) when the caller leaves it to the
    method.  The section fixes only the well-scaled case; the reading taken
    here: the power of two that puts max|X| / s1 in [2^14, 2^15), so the
    leading fp16 term keeps its 11 bits and stays a factor two below fp16's
    largest finite value; 1 when max|X| is 0 or not finite; never below
    2^-126 (the smallest normal fp32 power of two)."""
    x = np.asarray(x, dtype=np.float64)
    mx = float(np.max(np.abs(x))) if x.size else 0.0
    if mx == 0.0 or not np.isfinite(mx):
        return 1.0
    e = int(np.floor(np.log2(mx))) - 14
    return float(2.0 ** max(e, -126))


def gemm_split3(layout: str, a: np.ndarray, b: np.ndarray, a_scale: float, b_scale: float,
                alpha: float = 1.0, beta: float = 0.0, c: Optional[np.ndarray] = None) -> np.ndarray:
    """alpha * (a1 b1 A1B1 + a1 b2 A1B2 + a2 b1 A2B1) + beta * C, exactly, for
    the Eq. (1) splits of A (scale a1) and B (scale b1)."""
    a1, a2 = split_f16(a, a_scale)
    b1, b2 = split_f16(b, b_scale)
    sa2, sb2 = a_scale * SPLIT_SHIFT, b_scale * SPLIT_SHIFT
    prod = (a_scale * b_scale) * gemm(layout, a1, b1) + (a_scale * sb2) * gemm(layout, a1, b2) + \
        (sa2 * b_scale) * gemm(layout, a2, b1)
    return _axpby(alpha, prod, beta, c)


def _axpby(alpha: float, x: np.ndarray, beta: float, c: Optional[np.ndarray]) -> np.ndarray:
    return alpha * x + beta * c if beta != 0.0 else alpha * x


# ---------------------------------------------------------------------------
# Bias + ReLU epilogue and its backward (a fully connected / convolution
# layer's activation; section 2.1 backpropagation).
# ReLU keeps NaN (x < 0 is false for NaN); its derivative at 0 is 0 and the
# mask is taken from the *stored* output: d/dz relu = [y_stored > 0], applied
# as a selection (masked entries are 0 even where the incoming value is inf).
# ---------------------------------------------------------------------------

def relu(z: np.ndarray) -> np.ndarray:
    return np.where(z < 0.0, 0.0, z)


def bias_act(x: np.ndarray, bias: Optional[np.ndarray], act: str) -> np.ndarray:
    z = x if bias is None else x + bias
    return relu(z) if act == "relu" else z


def relu_mask(y_stored: np.ndarray) -> np.ndarray:
    return (y_stored > 0.0).astype(np.float64)


def bias_act_bwd(dy: np.ndarray, y: Optional[np.ndarray], act: str) -> Tuple[np.ndarray, np.ndarray]:
    """dz = dy * [y > 0] (relu) or dy; db = column sums of dz.  The bracket is
    a selection: where y <= 0 the result is 0 even if dy is inf or NaN."""
    dz = np.where(y > 0.0, dy, 0.0) if act == "relu" else dy
    return dz, dz.sum(axis=0)


# ---------------------------------------------------------------------------
# 2-D convolution, stride 1, zero padding, NHWC x [Cout,R,S,Cin].
#   y[n,ho,wo,k]  = sum_{r,s,c} x[n, ho+r-p, wo+s-p, c] * w[k,r,s,c]
#   dx[n,h,w,c]   = sum_{k,r,s} dy[n, h-r+p, w-s+p, k] * w[k,r,s,c]
#   dw[k,r,s,c]   = sum_{n,ho,wo} dy[n,ho,wo,k] * x[n, ho+r-p, wo+s-p, c]
# (indices outside the image contribute zero).  Output size
# Ho = H + 2p - R + 1, Wo = W + 2p - S + 1.  The channel sum of each tap is a
# library matmul; the taps are summed in order.
# ---------------------------------------------------------------------------

def conv_out_hw(h: int, w: int, r: int, s: int, pad: int) -> Tuple[int, int]:
    return h + 2 * pad - r + 1, w + 2 * pad - s + 1


def _pad_hw(x: np.ndarray, pad: int) -> np.ndarray:
    return np.pad(x, ((0, 0), (pad, pad), (pad, pad), (0, 0)))


def conv2d_fwd(x: np.ndarray, w: np.ndarray, pad: int) -> np.ndarray:
    n, h, wd, c = x.shape
    k, r, s, c2 = w.shape
    assert c == c2
    ho, wo = conv_out_hw(h, wd, r, s, pad)
    xp = _pad_hw(x, pad)
    y = np.zeros((n, ho, wo, k))
    for i in range(r):
        for j in range(s):
            y += xp[:, i:i + ho, j:j + wo, :] @ w[:, i, j, :].T
    return y


def conv2d_bwd_data(dy: np.ndarray, w: np.ndarray, pad: int, h: int, wd: int) -> np.ndarray:
    n, ho, wo, k = dy.shape
    k2, r, s, c = w.shape
    assert k == k2
    dx = np.zeros((n, h, wd, c))
    for i in range(r):
        for j in range(s):
            # output pixel (ho', wo') reads input pixel (ho'+i-p, wo'+j-p)
            h0, h1 = max(0, pad - i), min(ho, h + pad - i)
            w0, w1 = max(0, pad - j), min(wo, wd + pad - j)
            if h0 >= h1 or w0 >= w1:
                continue
            dx[:, h0 + i - pad:h1 + i - pad, w0 + j - pad:w1 + j - pad, :] += \
                dy[:, h0:h1, w0:w1, :] @ w[:, i, j, :]
    return dx


def conv2d_bwd_filter(x: np.ndarray, dy: np.ndarray, pad: int, r: int, s: int) -> np.ndarray:
    n, h, wd, c = x.shape
    n2, ho, wo, k = dy.shape
    assert n == n2
    xp = _pad_hw(x, pad)
    dym = dy.reshape(-1, k)
    dw = np.zeros((k, r, s, c))
    for i in range(r):
        for j in range(s):
            dw[:, i, j, :] = dym.T @ xp[:, i:i + ho, j:j + wo, :].reshape(-1, c)
    return dw


# ---------------------------------------------------------------------------
# 2x2 stride-2 max pooling (NHWC).  The window is scanned in row-major order
# (0:(0,0) 1:(0,1) 2:(1,0) 3:(1,1)); the first maximum wins (strict >), and
# the backward pass routes each gradient to that position only.
# ---------------------------------------------------------------------------

def maxpool2_fwd(x: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    n, h, w, c = x.shape
    cand = [x[:, di:h - h % 2:2, dj:w - w % 2:2, :] for di in (0, 1) for dj in (0, 1)]
    y = cand[0].copy()
    arg = np.zeros(y.shape, dtype=np.uint8)
    for idx in (1, 2, 3):
        better = cand[idx] > y
        y = np.where(better, cand[idx], y)
        arg = np.where(better, np.uint8(idx), arg)
    return y, arg


def maxpool2_bwd(dy: np.ndarray, arg: np.ndarray, h: int, w: int) -> np.ndarray:
    n, ho, wo, c = dy.shape
    dx = np.zeros((n, h, w, c))
    for idx in range(4):
        di, dj = divmod(idx, 2)
        dx[:, di:2 * ho:2, dj:2 * wo:2, :] = np.where(arg == idx, dy, 0.0)
    return dx


# ---------------------------------------------------------------------------
# Losses.  Mean over the batch; the gradient is multiplied by the loss scale S
# (S = 1 without loss scaling) and divided by B.
# ---------------------------------------------------------------------------

def softmax_xent(z: np.ndarray, labels: np.ndarray, scale: float = 1.0) -> Tuple[float, np.ndarray]:
    """L = -(1/B) sum_i log softmax(z_i)[y_i]  (max-subtracted log-sum-exp);
    dz = S * (softmax(z) - onehot(y)) / B.  A label outside [0, C) makes the
    loss and that row of dz NaN."""
    b, c = z.shape
    m = z.max(axis=1, keepdims=True)
    lse = m + np.log(np.exp(z - m).sum(axis=1, keepdims=True))
    logp = z - lse
    p = np.exp(logp)
    lab = np.asarray(labels).astype(np.int64)
    ok = (lab >= 0) & (lab < c)
    onehot = np.zeros_like(z)
    onehot[np.arange(b)[ok], lab[ok]] = 1.0
    picked = np.where(ok, logp[np.arange(b), np.where(ok, lab, 0)], np.nan)
    loss = -picked.sum() / b
    dz = scale * (p - onehot) / b
    dz[~ok, :] = np.nan
    return float(loss), dz


def mse_loss(y: np.ndarray, t: np.ndarray, scale: float = 1.0) -> Tuple[float, np.ndarray]:
    """L = (1/B) sum_{i,j} (y - t)^2 ;  dy = S * 2 (y - t) / B."""
    b = y.shape[0]
    d = y - t
    return float((d * d).sum() / b), scale * 2.0 * d / b


# ---------------------------------------------------------------------------
# Minibatch SGD (section 3.1) with heavy-ball momentum and a dynamic loss
# scaler.  Momentum and loss scaling are part of the workloads, not of the
# paper.  Scaler: overflow = any non-finite gradient element; on overflow the
# whole update is skipped and S <- max(S * backoff, min_scale), good_steps = 0;
# otherwise g <- g / S is applied and after ``growth_interval`` consecutive good
# steps S <- S * growth.
# ---------------------------------------------------------------------------

def new_scaler(scale: float, growth_interval: int = 2000, growth: float = 2.0,
               backoff: float = 0.5, min_scale: float = 1.0) -> dict:
    return dict(scale=float(scale), good_steps=0, overflow=0, growth_interval=growth_interval,
                growth=growth, backoff=backoff, min_scale=min_scale)


def sgd_update(w: np.ndarray, g: np.ndarray, v: Optional[np.ndarray], lr: float,
               momentum: float, scaler: Optional[dict]):
    """Returns (w, v, scaler, applied).  Inputs are not modified."""
    w = w.copy()
    v = None if v is None else v.copy()
    sc = None if scaler is None else dict(scaler)
    s = 1.0
    if sc is not None:
        if not np.all(np.isfinite(g)):
            sc["overflow"] = 1
            sc["scale"] = max(sc["scale"] * sc["backoff"], sc["min_scale"])
            sc["good_steps"] = 0
            return w, v, sc, False
        sc["overflow"] = 0
        s = sc["scale"]
    gs = g / s
    if v is not None:
        v = momentum * v + gs
        w = w - lr * v
    else:
        w = w - lr * gs
    if sc is not None:
        sc["good_steps"] += 1
        if sc["good_steps"] >= sc["growth_interval"]:
            sc["scale"] = sc["scale"] * sc["growth"]
            sc["good_steps"] = 0
    return w, v, sc, True
