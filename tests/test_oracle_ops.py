"""Pins for the oracle's building blocks: brute force, torch CPU library calls, round trips."""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import ops
from oracle import codec_float as cf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rng(seed=0):
    return np.random.default_rng(seed)


def t64(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))


def test_pixel_unshuffle_hand_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "pixel_unshuffle_4x4.json")))
    x = np.array(g["input"], dtype=np.float64)[None]
    out = ops.pixel_unshuffle(x, g["r"])
    np.testing.assert_array_equal(out, np.array(g["output"], dtype=np.float64))
    np.testing.assert_array_equal(ops.pixel_shuffle(out, g["r"]), x)


@pytest.mark.parametrize("shape,r", [((3, 16, 24), 8), ((5, 8, 4), 2), ((2, 6, 9), 3)])
def test_pixel_shuffle_round_trip_and_torch(shape, r):
    x = rng(1).standard_normal(shape)
    u = ops.pixel_unshuffle(x, r)
    np.testing.assert_array_equal(ops.pixel_shuffle(u, r), x)
    np.testing.assert_array_equal(u, F.pixel_unshuffle(t64(x)[None], r)[0].numpy())
    np.testing.assert_array_equal(ops.pixel_shuffle(u, r), F.pixel_shuffle(t64(u)[None], r)[0].numpy())


def brute_conv1x1(x, w, b):
    K, H, W = x.shape
    out = np.zeros((w.shape[0], H, W))
    for n in range(w.shape[0]):
        for yy in range(H):
            for xx in range(W):
                acc = b[n]
                for k in range(K):
                    acc += w[n, k] * x[k, yy, xx]
                out[n, yy, xx] = acc
    return out


def brute_dw(x, w, b):
    C, H, W = x.shape
    out = np.zeros_like(x)
    for c in range(C):
        for yy in range(H):
            for xx in range(W):
                acc = b[c]
                for dy in (-1, 0, 1):
                    for dx in (-1, 0, 1):
                        sy, sx = yy + dy, xx + dx
                        if 0 <= sy < H and 0 <= sx < W:
                            acc += w[c, dy + 1, dx + 1] * x[c, sy, sx]
                out[c, yy, xx] = acc
    return out


def brute_conv2x2s2(x, w, b):
    C, H, W = x.shape
    out = np.zeros((w.shape[0], H // 2, W // 2))
    for o in range(w.shape[0]):
        for Y in range(H // 2):
            for X in range(W // 2):
                acc = b[o]
                for c in range(C):
                    for i in range(2):
                        for j in range(2):
                            acc += w[o, c, i, j] * x[c, 2 * Y + i, 2 * X + j]
                out[o, Y, X] = acc
    return out


def test_conv1x1_brute_force_and_torch():
    r = rng(2)
    x = r.standard_normal((6, 4, 5))
    w = r.standard_normal((7, 6))
    b = r.standard_normal(7)
    got = ops.conv1x1(x, w, b)
    np.testing.assert_allclose(got, brute_conv1x1(x, w, b), rtol=0, atol=1e-12)
    ref = F.conv2d(t64(x)[None], t64(w)[:, :, None, None], t64(b))[0].numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_dwconv3x3_brute_force_and_torch():
    r = rng(3)
    x = r.standard_normal((4, 5, 7))
    w = r.standard_normal((4, 3, 3))
    b = r.standard_normal(4)
    got = ops.dwconv3x3(x, w, b)
    np.testing.assert_allclose(got, brute_dw(x, w, b), rtol=0, atol=1e-12)
    ref = F.conv2d(t64(x)[None], t64(w)[:, None], t64(b), padding=1, groups=4)[0].numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_dwconv3x3_single_pixel_and_impulse():
    # 1x1 image: only the centre tap sees data; impulse response reproduces the flipped kernel.
    w = np.arange(9, dtype=np.float64).reshape(1, 3, 3)
    got = ops.dwconv3x3(np.full((1, 1, 1), 2.0), w, np.zeros(1))
    assert got[0, 0, 0] == 2.0 * w[0, 1, 1]
    imp = np.zeros((1, 5, 5))
    imp[0, 2, 2] = 1.0
    resp = ops.dwconv3x3(imp, w, np.zeros(1))
    np.testing.assert_array_equal(resp[0, 1:4, 1:4], w[0, ::-1, ::-1])


def test_conv2x2s2_brute_force_and_torch():
    r = rng(4)
    x = r.standard_normal((3, 4, 6))
    w = r.standard_normal((5, 3, 2, 2))
    b = r.standard_normal(5)
    got = ops.conv2x2s2(x, w, b)
    np.testing.assert_allclose(got, brute_conv2x2s2(x, w, b), rtol=0, atol=1e-12)
    ref = F.conv2d(t64(x)[None], t64(w), t64(b), stride=2)[0].numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_leaky_relu_values():
    h = np.array([-2.0, -0.5, 0.0, 0.5, 3.0])
    np.testing.assert_array_equal(ops.leaky_relu(h, 0.1), [-0.2, -0.05, 0.0, 0.5, 3.0])


def test_patch_embed_equals_strided_conv():
    # unshuffle x8 + 1x1 == 8x8 stride-8 convolution with weight[o, c, i, j] = W[o, 64c + 8i + j]
    r = rng(5)
    x = r.uniform(0, 1, (3, 16, 24))
    W = r.standard_normal((4, 192))
    b = r.standard_normal(4)
    got = ops.conv1x1(ops.pixel_unshuffle(x, 8), W, b)
    ref = F.conv2d(t64(x)[None], t64(W.reshape(4, 3, 8, 8)), t64(b), stride=8)[0].numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_upsample_equals_transposed_conv():
    # 1x1 C->4C + pixel-shuffle x2 == 2x2 stride-2 transposed conv, weight[c_in, c, i, j] = W[4c+2i+j, c_in]
    r = rng(6)
    C = 3
    y = r.standard_normal((C, 3, 4))
    W = r.standard_normal((4 * C, C))
    b = r.standard_normal(4 * C)
    got = ops.pixel_shuffle(ops.conv1x1(y, W, b), 2)
    wt = W.reshape(C, 2, 2, C).transpose(3, 0, 1, 2)
    ref = F.conv_transpose2d(t64(y)[None], t64(wt), None, stride=2)[0].numpy()
    # bias of the sub-position (i, j) of channel c is b[4c+2i+j]
    bias_map = np.zeros((C, 6, 8))
    for c in range(C):
        for i in range(2):
            for j in range(2):
                bias_map[c, i::2, j::2] = b[4 * c + 2 * i + j]
    np.testing.assert_allclose(got, ref + bias_map, rtol=0, atol=1e-12)


def test_reconstruction_equals_transposed_conv():
    r = rng(7)
    C = 4
    f = r.standard_normal((C, 2, 3))
    W = r.standard_normal((192, C)) * 0.1
    b = np.zeros(192)
    got = ops.pixel_shuffle(ops.conv1x1(f, W, b), 8)
    wt = W.reshape(3, 8, 8, C).transpose(3, 0, 1, 2)
    ref = F.conv_transpose2d(t64(f)[None], t64(wt), None, stride=8)[0].numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def test_dc_block_matches_torch_composition():
    r = rng(8)
    C = 6

    class P:  # minimal stand-in with the oracle's field names
        pass

    blk = P()
    blk.dw, blk.pw1, blk.pw2 = P(), P(), P()
    blk.kind = "lrelu"
    blk.dw.w, blk.dw.b = r.standard_normal((C, 3, 3)), r.standard_normal(C)
    blk.pw1.w, blk.pw1.b = r.standard_normal((2 * C, C)), r.standard_normal(2 * C)
    blk.pw2.w, blk.pw2.b = r.standard_normal((C, 2 * C)), r.standard_normal(C)
    z = r.standard_normal((C, 5, 4))
    got = cf.dc_block(z, blk)
    tz = t64(z)[None]
    a = F.conv2d(tz, t64(blk.dw.w)[:, None], t64(blk.dw.b), padding=1, groups=C)
    h = F.conv2d(a, t64(blk.pw1.w)[:, :, None, None], t64(blk.pw1.b))
    g = F.leaky_relu(h, 0.1)
    ref = (tz + F.conv2d(g, t64(blk.pw2.w)[:, :, None, None], t64(blk.pw2.b)))[0].numpy()
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)
