"""Pins of the oracle's two-step entropy model with the hyper latent z
(Sec. 4.4; supplementary "Entropy model", "Parallel Coding").

* Parameter list: counts and shapes against the generator's list.
* Reduction: with the hyper and second-step convolutions zero the model is the
  one-step model of codec_float / codec_int (same symbols, latent, context,
  y rate), and every z symbol is 0, whose rate is the closed form
  -log2 erf(1 / (2 sqrt2 sigma_z)) per element.
* Brute force: the entropy step on a small latent evaluated element by element
  with nested loops (float64) and with Python integers and Fraction rounding
  (the integer path, Alg. 1 for every convolution).
* The decoder's order (z, distribution, y^1, y^2) reproduces the encoder's
  latent exactly.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth
from oracle import codec_float as cf
from oracle import codec_int as ci
from oracle import hyperprior as hp
from oracle.params import CZ


def hyper_params(C=8, ne=1, nd=1, zero_hyper=False):
    flat = synth.make_weights(C, ne, nd, hyper=True)
    p = oracle.unpack(flat, C, ne, nd, hyper=True)
    if zero_hyper:
        h = p.hyper
        for c in (h.zana, h.zsyn, h.step2):
            c.w[...] = 0.0
            c.b[...] = 0.0
    return p


def test_parameter_list():
    for C in (64, 128, 256):
        n = sum(int(np.prod(s)) for _, s, _, _ in synth.param_list(C, 2, 3, hyper=True))
        assert n == oracle.params.count(C, 2, 3, hyper=True)
        assert n - oracle.params.count(C, 2, 3) == CZ * 4 * C + CZ + 8 * C * CZ + 8 * C + C * C // 2 + C + 64 * CZ
    p = hyper_params(16)
    assert p.hyper.zana.w.shape == (CZ, 16, 2, 2) and p.hyper.zsyn.w.shape == (128, CZ)
    assert p.hyper.step2.w.shape == (16, 8) and p.hyper.zbank.shape == (64, CZ)
    assert (p.hyper.zbank > 0).all()


def test_nearest_bank_row():
    assert [hp.z_row(q) for q in (0, 0.49, 0.5, 1.2, 62.5, 63)] == [0, 0, 1, 1, 63, 63]
    with pytest.raises(ValueError):
        hp.z_row(63.5)


def test_reduces_to_one_step_model_float():
    p = hyper_params(64, 2, 2, zero_hyper=True)
    x = next(synth.frame_sequence("tiny"))
    st = cf.State(np.random.default_rng(1).normal(0, 1, (64, 8, 8)), np.random.default_rng(2).normal(0, 2, (64, 4, 4)))
    r = hp.encode_frame_float(p, x, st)
    one = cf.encode_frame(p, x, st)
    np.testing.assert_array_equal(r.sym.y(), one.q)
    np.testing.assert_array_equal(r.state.yhat, one.state.yhat)
    np.testing.assert_array_equal(r.state.feat, one.state.feat)
    assert r.bits_y1 + r.bits_y2 == pytest.approx(one.bits, rel=1e-12)
    assert not r.sym.qz.any()
    sz = hp.z_sigma(p, 0)
    ref = 4 * sum(-math.log2(math.erf(1.0 / (2.0 * math.sqrt(2.0) * s))) for s in sz)  # 2 x 2 z positions
    assert r.bits_z == pytest.approx(ref, rel=1e-12)


def test_reduces_to_one_step_model_int():
    p = hyper_params(64, 2, 2, zero_hyper=True)
    ip, ih = ci.integerize(p), hp.integerize_hyper(p)
    x = next(synth.frame_sequence("tiny"))
    rng = np.random.default_rng(3)
    st = ci.State(rng.integers(-2000, 2000, (64, 8, 8)), rng.integers(-3000, 3000, (64, 4, 4)))
    r = hp.encode_frame_int(p, ip, ih, x, st)
    one = ci.encode_frame(ip, x, st)
    np.testing.assert_array_equal(r.sym.y(), one.q)
    np.testing.assert_array_equal(r.state.yhat, one.state.yhat)
    np.testing.assert_array_equal(r.state.feat, one.state.feat)
    assert r.bits_y1 + r.bits_y2 == pytest.approx(one.bits, rel=1e-12)


def _brute_float(p, y, yhat_prev):
    """Nested-loop evaluation of the float entropy step."""
    C = p.C
    H2 = C // 2
    h16, w16 = y.shape[1:]
    h32, w32 = h16 // 2, w16 // 2
    hz = p.hyper
    z = np.zeros((CZ, h32, w32))
    for o in range(CZ):
        for Y in range(h32):
            for X in range(w32):
                acc = hz.zana.b[o]
                for c in range(C):
                    for i in range(2):
                        for j in range(2):
                            acc += hz.zana.w[o, c, i, j] * y[c, 2 * Y + i, 2 * X + j]
                z[o, Y, X] = acc
    qz = np.vectorize(round)(z).astype(np.float64)  # Python round: half to even
    hpar = np.zeros((2 * C, h16, w16))
    for m in range(2 * C):
        for Y in range(h32):
            for X in range(w32):
                for i in range(2):
                    for j in range(2):
                        r = 4 * m + 2 * i + j
                        hpar[m, 2 * Y + i, 2 * X + j] = hz.zsyn.b[r] + sum(hz.zsyn.w[r, k] * qz[k, Y, X] for k in range(CZ))
    ms = np.zeros((2 * C, h16, w16))
    for r in range(2 * C):
        for Y in range(h16):
            for X in range(w16):
                ms[r, Y, X] = p.head.b[r] + sum(p.head.w[r, k] * yhat_prev[k, Y, X] for k in range(C)) + hpar[r, Y, X]
    q1 = np.vectorize(round)(y[:H2] - ms[:H2]).astype(np.float64)
    yhat1 = q1 + ms[:H2]
    d = np.zeros((C, h16, w16))
    for r in range(C):
        for Y in range(h16):
            for X in range(w16):
                d[r, Y, X] = hz.step2.b[r] + sum(hz.step2.w[r, k] * yhat1[k, Y, X] for k in range(H2))
    mu2 = ms[H2:C] + d[:H2]
    q2 = np.vectorize(round)(y[H2:] - mu2).astype(np.float64)
    return qz, q1, q2, np.concatenate([yhat1, q2 + mu2]), ms[C:C + H2], ms[C + H2:] + d[H2:]


def test_float_entropy_step_brute_force():
    p = hyper_params(8)
    rng = np.random.default_rng(4)
    y = rng.normal(0, 3, (8, 4, 6))
    yp = rng.normal(0, 3, (8, 4, 6))
    sym, yhat, s1, s2 = hp.two_step_float(p, y, yp)
    qz, q1, q2, yh, sa, sb = _brute_float(p, y, yp)
    assert np.abs(qz).max() > 0  # z is not trivially zero
    np.testing.assert_array_equal(sym.qz, qz)
    np.testing.assert_array_equal(sym.q1, q1)
    np.testing.assert_array_equal(sym.q2, q2)
    np.testing.assert_allclose(yhat, yh, rtol=0, atol=1e-12)
    np.testing.assert_allclose(s1, oracle.sigma_from_s(sa), rtol=1e-12)
    np.testing.assert_allclose(s2, oracle.sigma_from_s(sb), rtol=1e-12)


def _brute_int(ip, ih, y, yhat_prev):
    """Python-integer evaluation of the integer entropy step (Alg. 1 with
    Fraction round-half-even for every rescale, saturating adds)."""
    C = ip.C
    H2 = C // 2
    h16, w16 = y.shape[1:]

    def rq(a, s):
        return round(Fraction(int(a), 1 << s))

    def c16(v):
        return max(-32768, min(32767, v))

    def conv_el(w_row, b, xs):
        return c16(rq(sum(int(a) * int(b_) for a, b_ in zip(w_row, xs)) + 512 * int(b), 13))

    zq = np.zeros((CZ, h16 // 2, w16 // 2), np.int64)
    for o in range(CZ):
        for Y in range(h16 // 2):
            for X in range(w16 // 2):
                ws, xs = [], []
                for c in range(C):
                    for i in range(2):
                        for j in range(2):
                            ws.append(ih.zana.w[o, c, i, j])
                            xs.append(y[c, 2 * Y + i, 2 * X + j])
                zq[o, Y, X] = rq(conv_el(ws, ih.zana.b[o], xs), 9)
    zhat = np.vectorize(lambda v: c16(512 * int(v)))(zq)
    mu = np.zeros((2 * C, h16, w16), np.int64)
    for r in range(2 * C):
        for Y in range(h16):
            for X in range(w16):
                head = conv_el(ip.head.w[r], ip.head.b[r], yhat_prev[:, Y, X])
                row = 4 * r + 2 * (Y % 2) + (X % 2)   # pixel shuffle x2: channel r at (2Y' + i, 2X' + j)
                hyp = conv_el(ih.zsyn.w[row], ih.zsyn.b[row], zhat[:, Y // 2, X // 2])
                mu[r, Y, X] = c16(head + hyp)
    q1 = np.vectorize(lambda v: rq(v, 9))(y[:H2] - mu[:H2])
    yhat1 = np.vectorize(c16)(512 * q1 + mu[:H2])
    out = np.zeros((C, h16, w16), np.int64)
    for r in range(C):
        for Y in range(h16):
            for X in range(w16):
                out[r, Y, X] = conv_el(ih.step2.w[r], ih.step2.b[r], yhat1[:, Y, X])
    mu2 = np.vectorize(c16)(mu[H2:C] + out[:H2])
    s2 = np.vectorize(c16)(mu[C + H2:] + out[H2:])
    q2 = np.vectorize(lambda v: rq(v, 9))(y[H2:] - mu2)
    yhat2 = np.vectorize(c16)(512 * q2 + mu2)
    return zq, q1, q2, np.concatenate([yhat1, yhat2]), mu[C:C + H2], s2


def test_int_entropy_step_brute_force():
    p = hyper_params(8)
    ip, ih = ci.integerize(p), hp.integerize_hyper(p)
    rng = np.random.default_rng(5)
    y = rng.integers(-4000, 4000, (8, 4, 6))
    yp = rng.integers(-4000, 4000, (8, 4, 6))
    sym, yhat, s1, s2 = hp.two_step_int(ip, ih, y, yp)
    zq, q1, q2, yh, sa, sb = _brute_int(ip, ih, y, yp)
    assert np.abs(zq).max() > 0
    np.testing.assert_array_equal(sym.qz, zq)
    np.testing.assert_array_equal(sym.q1, q1)
    np.testing.assert_array_equal(sym.q2, q2)
    np.testing.assert_array_equal(yhat, yh)
    np.testing.assert_allclose(s1, ci.sigma_int(sa), rtol=1e-15)
    np.testing.assert_allclose(s2, ci.sigma_int(sb), rtol=1e-15)


@pytest.mark.parametrize("path", ["fp16", "int16"])
def test_decoder_order_reproduces_encoder(path):
    C = 64
    p = hyper_params(C, 2, 2)
    frames = list(synth.frame_sequence("tiny", 3))
    if path == "fp16":
        st_e = st_d = cf.zero_state(p, 64, 64)
        for x in frames:
            r = hp.encode_frame_float(p, x, st_e)
            xh, st_d = hp.decode_frame_float(p, r.sym, st_d)
            np.testing.assert_array_equal(st_d.yhat, r.state.yhat)
            np.testing.assert_array_equal(st_d.feat, r.state.feat)
            st_e = r.state
    else:
        ip, ih = ci.integerize(p), hp.integerize_hyper(p)
        st_e = st_d = ci.zero_state(ip, 64, 64)
        for x in frames:
            r = hp.encode_frame_int(p, ip, ih, x, st_e)
            xh, st_d = hp.decode_frame_int(ip, ih, r.sym, st_d)
            np.testing.assert_array_equal(st_d.yhat, r.state.yhat)
            np.testing.assert_array_equal(st_d.feat, r.state.feat)
            _, s1, s2 = hp.latent_from_symbols_int(ip, ih, r.sym, st_e.yhat)
            np.testing.assert_array_equal(s1, r.sigma1)
            np.testing.assert_array_equal(s2, r.sigma2)
            st_e = r.state
