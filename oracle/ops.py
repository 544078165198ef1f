"""Plain float64 building blocks of the transform, planar (C, H, W) layout.

Each is the textbook definition; pins live in ``tests/test_oracle_ops.py``
(nested-loop brute force, ``torch.nn.functional`` on CPU, round trips).
"""
from __future__ import annotations

import numpy as np
from scipy.special import expit


def pixel_unshuffle(x: np.ndarray, r: int) -> np.ndarray:
    """Patch embedding's space-to-depth (Sec. 4.1, Fig. 4 "patch embedding").

    out[c*r*r + i*r + j, y, x] = x[c, r*y + i, r*x + j].
    """
    C, H, W = x.shape
    assert H % r == 0 and W % r == 0
    return (x.reshape(C, H // r, r, W // r, r)
             .transpose(0, 2, 4, 1, 3)
             .reshape(C * r * r, H // r, W // r))


def pixel_shuffle(v: np.ndarray, r: int) -> np.ndarray:
    """Inverse of :func:`pixel_unshuffle`: out[c, r*y+i, r*x+j] = v[c*r*r + i*r + j, y, x]."""
    Cr, h, w = v.shape
    assert Cr % (r * r) == 0
    C = Cr // (r * r)
    return (v.reshape(C, r, r, h, w)
             .transpose(0, 3, 1, 4, 2)
             .reshape(C, h * r, w * r))


def conv1x1(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Pointwise convolution: out[n] = sum_k w[n, k] x[k] + b[n]."""
    K, h, wd = x.shape
    assert w.shape[1] == K
    out = w @ x.reshape(K, h * wd) + b[:, None]
    return out.reshape(w.shape[0], h, wd)


def dwconv3x3(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Depthwise 3x3 cross-correlation, zero padding 1 (the DC block's depth-wise conv, Supp. B.1).

    out[c, y, x] = sum_{dy,dx in -1..1} w[c, dy+1, dx+1] * x[c, y+dy, x+dx] + b[c].
    """
    C, H, W = x.shape
    pad = np.zeros((C, H + 2, W + 2), dtype=np.float64)
    pad[:, 1:H + 1, 1:W + 1] = x
    out = np.zeros((C, H, W), dtype=np.float64)
    for ky in range(3):
        for kx in range(3):
            out += w[:, ky, kx][:, None, None] * pad[:, ky:ky + H, kx:kx + W]
    return out + b[:, None, None]


def conv2x2s2(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """2x2 convolution, stride 2, no padding.

    out[o, Y, X] = sum_{c,i,j} w[o, c, i, j] * x[c, 2Y+i, 2X+j] + b[o].
    """
    C, H, W = x.shape
    assert H % 2 == 0 and W % 2 == 0 and w.shape[1:] == (C, 2, 2)
    out = np.zeros((w.shape[0], (H // 2) * (W // 2)), dtype=np.float64)
    for i in range(2):
        for j in range(2):
            out += w[:, :, i, j] @ x[:, i::2, j::2].reshape(C, -1)
    return (out + b[:, None]).reshape(w.shape[0], H // 2, W // 2)


def leaky_relu(h: np.ndarray, slope: float = 0.1) -> np.ndarray:
    return np.where(h >= 0.0, h, slope * h)


def wsilu(x: np.ndarray, alpha: float = 4.0) -> np.ndarray:
    """Weighted SiLU of Supp. B.1: x * sigmoid(alpha x), alpha = 4 by default."""
    return x * expit(alpha * x)
