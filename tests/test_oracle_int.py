"""Pins for the integerised oracle: printed constants, exact rounding, exact integer products."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import codec_int as ci

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_printed_fixed_point_constants():
    g = json.load(open(os.path.join(GOLDEN, "fixed_point.json")))
    assert ci.K1 == g["K1"] and (1 << ci.K2_SHIFT) == g["K2"]
    assert ci.frame_to_int(np.array([1.0]))[0] == g["float_one_maps_to"]
    lo, hi = g["int16_range"]
    assert (ci.INT16_MIN, ci.INT16_MAX) == (lo, hi)
    # the int16 range maps to [-64.0, 63.998...] (printed to 3 decimals)
    assert lo / ci.K1 == g["float_range_printed"][0]
    assert round(hi / ci.K1, 3) == g["float_range_printed"][1]
    assert ci.LRELU_SLOPE_I == round(0.1 * g["K2"])


def test_rhe_shift_exhaustive_window_against_fraction():
    a = np.arange(-70000, 70001, dtype=np.int64)
    for s in (1, 2, 9, 13):
        got = ci.rhe_shift(a, s)
        ref = np.array([round(Fraction(int(v), 1 << s)) for v in a[::7]], dtype=np.int64)
        np.testing.assert_array_equal(got[::7], ref)
        # every tie in the window rounds to even
        ties = a[(a % (1 << s)) == (1 << (s - 1))]
        assert np.all(ci.rhe_shift(ties, s) % 2 == 0)


def test_rhe_shift_random_int32_against_rint():
    r = np.random.default_rng(0)
    a = r.integers(-(1 << 31), 1 << 31, size=200000, dtype=np.int64)
    for s in (9, 13):
        np.testing.assert_array_equal(ci.rhe_shift(a, s), np.rint(a / float(1 << s)).astype(np.int64))


def test_int_matmul_exact_against_python_ints():
    r = np.random.default_rng(1)
    for K in (1, 7, 64, 1024):
        w = r.integers(-32768, 32768, size=(5, K), dtype=np.int64)
        x = r.integers(-32768, 32768, size=(K, 3), dtype=np.int64)
        ref = np.array([[sum(int(w[i, k]) * int(x[k, j]) for k in range(K)) for j in range(3)] for i in range(5)], dtype=object)
        got = ci.int_matmul(w, x)
        assert all(int(got[i, j]) == ref[i, j] for i in range(5) for j in range(3))


def test_int_conv_follows_algorithm_1_brute_force():
    # y_i = clip(round((sum x_i w_i + b_i K1) / K2)) with Python integers and Fractions
    r = np.random.default_rng(2)
    w_f = (r.standard_normal((3, 4)) * 0.3).astype(np.float16).astype(np.float64)
    b_f = r.uniform(-0.1, 0.1, 3).astype(np.float16).astype(np.float64)
    x_i = r.integers(-4000, 4000, size=(4, 2, 2), dtype=np.int64)
    c = ci.IConv(ci.quantize_param(w_f), ci.quantize_param(b_f))
    got = ci.int_conv1x1(x_i, c)
    for n in range(3):
        wi = [round(Fraction(float(v)) * 8192) for v in w_f[n]]
        bi = round(Fraction(float(b_f[n])) * 8192)
        for yy in range(2):
            for xx in range(2):
                a = sum(wi[k] * int(x_i[k, yy, xx]) for k in range(4)) + bi * 512
                ref = max(-32768, min(32767, round(Fraction(a, 8192))))
                assert got[n, yy, xx] == ref


def test_int_conv_approximates_float_conv():
    from oracle import ops
    r = np.random.default_rng(3)
    w_f = (r.standard_normal((8, 16)) / 4).astype(np.float16).astype(np.float64)
    b_f = r.uniform(-0.1, 0.1, 8).astype(np.float16).astype(np.float64)
    x_f = r.uniform(-2, 2, (16, 3, 3))
    x_i = ci.clip16(np.rint(x_f * 512))
    y_i = ci.int_conv1x1(x_i, ci.IConv(ci.quantize_param(w_f), ci.quantize_param(b_f)))
    y_f = ops.conv1x1(x_i / 512.0, w_f, b_f)
    # error: weight rounding (<= 2^-14 per weight) x |x| summed, bias rounding, final rounding
    bound = 16 * 2.0 * 2 ** -14 + 2 ** -14 + 0.5 / 512 + 1e-12
    assert np.max(np.abs(y_i / 512.0 - y_f)) <= bound


def test_overflow_is_flagged():
    c = ci.IConv(np.full((1, 1024), 32000, dtype=np.int64), np.zeros(1, dtype=np.int64))
    x = np.full((1024, 1, 1), 32000, dtype=np.int64)
    with pytest.raises(OverflowError):
        ci.int_conv1x1(x, c)


def test_quantizer_properties():
    r = np.random.default_rng(4)
    y = r.integers(-20000, 20000, 100000, dtype=np.int64)
    mu = r.integers(-20000, 20000, 100000, dtype=np.int64)
    q, yhat = ci.quantize(y, mu)
    d = y - mu
    assert np.all(np.abs(d - 512 * q) <= 256)
    tie = np.abs(d - 512 * q) == 256
    assert np.all(q[tie] % 2 == 0)
    ok = np.abs(512 * q + mu) <= 32767
    np.testing.assert_array_equal(yhat[ok] - mu[ok], 512 * q[ok])


def test_int_leaky_relu():
    h = np.array([-32768, -8192, -5, -1, 0, 1, 32767], dtype=np.int64)
    g = ci.int_leaky_relu(h)
    assert list(g[4:]) == [0, 1, 32767]
    # 819 * -8192 / 8192 = -819 exactly; -5 * 819 / 8192 = -0.4999 -> 0; -32768 -> -3276
    assert g[1] == -819 and g[2] == 0 and g[3] == 0 and g[0] == -3276


def test_residual_saturates():
    assert list(ci.clip16(np.array([30000 + 5000, -30000 - 5000]))) == [32767, -32768]


def brute_int_lrelu_block(z, dw_w, dw_b, w1, b1, w2, b2):
    """The LeakyReLU DC block (reading A1) evaluated element by element with
    Python integers, every rescale an exact Fraction rounded half-to-even
    (Alg. 1: a = sum x_i w_i + b_i K1, y_i = clip(round(a / K2))), the negative
    branch of the LeakyReLU round(819 h / 8192), the residual a saturating
    int16 add of the block input and the clipped pw2 output."""
    C, H, W = z.shape

    def rq(num, den):
        return round(Fraction(int(num), int(den)))

    def c16(v):
        return max(-32768, min(32767, v))

    out = np.zeros_like(z)
    for y in range(H):
        for x in range(W):
            a = []
            for c in range(C):
                acc = 512 * int(dw_b[c])
                for dy in (-1, 0, 1):
                    for dx in (-1, 0, 1):
                        if 0 <= y + dy < H and 0 <= x + dx < W:
                            acc += int(dw_w[c, dy + 1, dx + 1]) * int(z[c, y + dy, x + dx])
                assert abs(acc) < 2 ** 31
                a.append(c16(rq(acc, 8192)))
            g = []
            for n in range(2 * C):
                acc = 512 * int(b1[n]) + sum(int(w1[n, k]) * a[k] for k in range(C))
                assert abs(acc) < 2 ** 31
                h = c16(rq(acc, 8192))
                g.append(h if h >= 0 else rq(819 * h, 8192))
            for n in range(C):
                acc = 512 * int(b2[n]) + sum(int(w2[n, k]) * g[k] for k in range(2 * C))
                assert abs(acc) < 2 ** 31
                p = c16(rq(acc, 8192))
                out[n, y, x] = c16(int(z[n, y, x]) + p)
    return out


def _int_block(dw_w, dw_b, w1, b1, w2, b2):
    return ci.IBlock(ci.IConv(dw_w, dw_b), ci.IConv(w1, b1), ci.IConv(w2, b2), "lrelu")


def test_int_lrelu_block_matches_brute_force():
    # the random-init block of the tiny configuration on a random int16 feature map
    import oracle
    import synth
    C = 8
    p = oracle.unpack(synth.make_weights(C, 1, 1), C, 1, 1)
    ib = ci.integerize(p).enc[0]
    rng = np.random.default_rng(11)
    z = rng.integers(-3000, 3000, size=(C, 5, 6), dtype=np.int64)
    got = ci.dc_block(z, ib)
    ref = brute_int_lrelu_block(z, ib.dw.w, ib.dw.b, ib.pw1.w, ib.pw1.b, ib.pw2.w, ib.pw2.b)
    np.testing.assert_array_equal(got, ref)


def test_int_lrelu_block_saturation_matches_brute_force():
    # Large weights and inputs near the int16 limits: the pw1 and pw2 rescales
    # clip (|a| / 8192 > 32767 while |a| < 2^31) and the residual add saturates
    # in both directions.  A clip placed before the residual add instead of
    # after it, or a missing clip of p, changes the result.
    C = 8
    rng = np.random.default_rng(12)
    dw_w = rng.integers(-4000, 4000, size=(C, 3, 3), dtype=np.int64)
    dw_b = rng.integers(-800, 800, size=C, dtype=np.int64)
    w1 = rng.integers(-16000, 16000, size=(2 * C, C), dtype=np.int64)
    b1 = rng.integers(-800, 800, size=2 * C, dtype=np.int64)
    w2 = rng.integers(-4000, 4000, size=(C, 2 * C), dtype=np.int64)
    b2 = rng.integers(-800, 800, size=C, dtype=np.int64)
    z = rng.integers(-32768, 32768, size=(C, 4, 5), dtype=np.int64)
    z[:, 0, :] = 32767
    z[:, 1, :] = -32768
    ib = _int_block(dw_w, dw_b, w1, b1, w2, b2)
    got = ci.dc_block(z, ib)
    ref = brute_int_lrelu_block(z, dw_w, dw_b, w1, b1, w2, b2)
    np.testing.assert_array_equal(got, ref)
    # the case is saturating: some pw1 / pw2 outputs and residual sums leave int16
    a = ci.int_dwconv3x3(z, ib.dw)
    h_acc = ci.int_matmul(w1, a.reshape(C, -1)) + 512 * b1[:, None]
    assert np.abs(ci.rhe_shift(h_acc, 13)).max() > 32767
    p = ci.int_conv1x1(ci.int_leaky_relu(ci.int_conv1x1(a, ib.pw1)), ib.pw2)
    assert (z + p > 32767).any() and (z + p < -32768).any()
    assert (np.abs(p) == 32767).any() or (p == -32768).any()
