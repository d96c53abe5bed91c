"""Winograd minimal filtering for 3x3 convolutions, F(2x2, 3x3), in fp64
(test infrastructure only).

Section 2.1 keeps the convolution algorithm swappable behind the layer; the
usual fast alternative for 3x3 filters is Winograd's minimal filtering
algorithm as applied to CNNs by Lavin and Gray ("Fast Algorithms for
Convolutional Neural Networks", 2016).  For a 4x4 input tile d and a 3x3
filter g it produces the 2x2 correlation output

    Y = A^T [ (G g G^T) (.) (B^T d B) ] A

((.) elementwise), with the transforms of F(2, 3) below.  Over channels the
elementwise product becomes 16 independent matrix products
M_xi[t, k] = sum_c V_xi[t, c] U_xi[k, c] (xi indexes the 4x4 transformed
positions, t the tiles), which is where the work goes.

The convolution it computes has a plain definition, ops.conv2d_fwd: that is
the oracle for the result.  This module states the algorithm (so tests can
check that it reproduces the definition, and derive the error bound of a
low-precision implementation from the magnitudes of its transformed values).
"""
from __future__ import annotations

import numpy as np

# F(2, 3): 2 outputs of a 3-tap correlation from 4 inputs with 4 products.
BT = np.array([[1.0, 0.0, -1.0, 0.0],
               [0.0, 1.0, 1.0, 0.0],
               [0.0, -1.0, 1.0, 0.0],
               [0.0, 1.0, 0.0, -1.0]])
G = np.array([[1.0, 0.0, 0.0],
              [0.5, 0.5, 0.5],
              [0.5, -0.5, 0.5],
              [0.0, 0.0, 1.0]])
AT = np.array([[1.0, 1.0, 1.0, 0.0],
               [0.0, 1.0, -1.0, -1.0]])


def tiles_hw(h: int, w: int, pad: int):
    """Output size (3x3 filter, stride 1) and the number of 2x2 output tiles."""
    ho, wo = h + 2 * pad - 2, w + 2 * pad - 2
    return ho, wo, -(-ho // 2), -(-wo // 2)


def filter_transform(w: np.ndarray) -> np.ndarray:
    """w [K, 3, 3, C] -> U [4, 4, K, C], U[:, :, k, c] = G w[k, :, :, c] G^T."""
    assert w.shape[1:3] == (3, 3)
    return np.einsum("ar,krsc,bs->abkc", G, w, G)


def input_tiles(x: np.ndarray, pad: int) -> np.ndarray:
    """x [N, H, W, C] -> d [N, TH, TW, 4, 4, C]: the 4x4 windows (stride 2) of
    the zero-padded input that the 2x2 output tiles read; rows and columns
    beyond the padded input (a ragged last tile) are zero."""
    n, h, w, c = x.shape
    ho, wo, th, tw = tiles_hw(h, w, pad)
    xp = np.zeros((n, 2 * th + 2, 2 * tw + 2, c))
    hh, ww = min(h, 2 * th + 2 - pad), min(w, 2 * tw + 2 - pad)
    xp[:, pad:pad + hh, pad:pad + ww, :] = x[:, :hh, :ww, :]
    d = np.zeros((n, th, tw, 4, 4, c))
    for a in range(4):
        for b in range(4):
            d[:, :, :, a, b, :] = xp[:, a:a + 2 * th:2, b:b + 2 * tw:2, :]
    return d


def _sandwich(left: np.ndarray, t: np.ndarray, right: np.ndarray) -> np.ndarray:
    """left @ t @ right^T over the two tile axes (3 and 4) of t [..., P, Q, C]."""
    s = np.tensordot(left, t, axes=([1], [3]))          # [a, N, TH, TW, Q, C]
    s = np.tensordot(right, s, axes=([1], [4]))         # [b, a, N, TH, TW, C]
    return np.moveaxis(np.moveaxis(s, 0, 4), 0, 3)      # [N, TH, TW, a, b, C]


def input_transform(d: np.ndarray) -> np.ndarray:
    """d [N, TH, TW, 4, 4, C] -> V = B^T d B, same shape."""
    return _sandwich(BT, d, BT)


def output_transform(m: np.ndarray) -> np.ndarray:
    """m [N, TH, TW, 4, 4, K] -> Y = A^T m A, [N, TH, TW, 2, 2, K]."""
    return _sandwich(AT, m, AT)


def products(v: np.ndarray, u: np.ndarray) -> np.ndarray:
    """M[..., a, b, k] = sum_c V[..., a, b, c] U[a, b, k, c]: the 16 matrix products."""
    m = np.empty(v.shape[:5] + (u.shape[2],))
    for a in range(4):
        for b in range(4):
            m[..., a, b, :] = v[..., a, b, :] @ u[a, b].T
    return m


def untile(yt: np.ndarray, ho: int, wo: int) -> np.ndarray:
    """[N, TH, TW, 2, 2, K] -> [N, HO, WO, K] (drops a ragged tile's extra row / column)."""
    n, th, tw, _, _, k = yt.shape
    return yt.transpose(0, 1, 3, 2, 4, 5).reshape(n, 2 * th, 2 * tw, k)[:, :ho, :wo, :]


def conv2d_fwd_winograd(x: np.ndarray, w: np.ndarray, pad: int) -> np.ndarray:
    """The 3x3 convolution (NHWC x KRSC, stride 1, zero padding) through
    F(2x2, 3x3): the four steps in order, in exact fp64 arithmetic."""
    n, h, wd, c = x.shape
    ho, wo, _, _ = tiles_hw(h, wd, pad)
    u = filter_transform(w)
    v = input_transform(input_tiles(x, pad))
    return untile(output_transform(products(v, u)), ho, wo)


def error_scale(x: np.ndarray, w: np.ndarray, pad: int) -> np.ndarray:
    """|A^T| ( sum_c |U| |V| ) |A| per output [N, HO, WO, K]: every rounding of
    a transformed operand or of a product sum in a Winograd implementation is
    relative to a term of this sum, so its error is a small multiple of it."""
    n, h, wd, c = x.shape
    ho, wo, _, _ = tiles_hw(h, wd, pad)
    u = np.abs(filter_transform(w))
    v = np.abs(input_transform(input_tiles(x, pad)))
    return untile(_sandwich(np.abs(AT), products(v, u), np.abs(AT)), ho, wo)
