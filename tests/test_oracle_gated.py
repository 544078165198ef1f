"""Pins of the gated DC-block form (Supp. B.1: WSiLU, Chunk; Sec. 4.5: the
sigmoid lookup table of the integer path).

* WSiLU against torch's SiLU (WSiLU(x) = SiLU(4x) / 4) and its reflection
  identity WSiLU(-x) = WSiLU(x) - x.
* The int16 sigmoid table against math.exp point by point, its symmetry
  S(v) + S(-v) = 512, monotonicity, saturation, and its distance from rounding
  ties (so that any exact evaluation gives the same table).
* The integer WSiLU and gate against exact rational rounding (fractions).
* The gated block, float and int, against nested-loop brute force on a tiny
  input, and the whole gated transform against torch convolutions.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth
from oracle import codec_float as cf
from oracle import codec_int as ci
from oracle import ops


def t64(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))


def test_wsilu_is_a_scaled_silu_and_reflects():
    x = np.linspace(-12, 12, 20001)
    ref = F.silu(t64(4.0 * x)).numpy() / 4.0
    np.testing.assert_allclose(ops.wsilu(x), ref, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(ops.wsilu(-x), ops.wsilu(x) - x, rtol=0, atol=1e-12)
    assert ops.wsilu(np.array([0.0]))[0] == 0.0


def test_sigmoid_table_definition_and_shape():
    S = ci.sigmoid_table()
    v = np.arange(-32768, 32768)
    assert S.shape == (65536,) and S.dtype == np.int64
    for vi in [-32768, -2000, -900, -513, -1, 0, 1, 7, 100, 512, 887, 32767]:
        want = 512.0 / (1.0 + math.exp(-4.0 * vi / 512.0))
        assert S[vi + 32768] == round(want)  # no ties (next test), so any rounding rule agrees
    assert S[32768] == 256
    assert np.all(np.diff(S) >= 0)
    np.testing.assert_array_equal(S[1:] + S[1:][::-1], 512)  # v and -v, v = -32767 .. 32767
    assert np.all(S[v >= 900] == 512) and np.all(S[v <= -900] == 0)


def test_sigmoid_table_has_no_rounding_ties():
    v = np.arange(-32768, 32768, dtype=np.float64)
    t = 512.0 / (1.0 + np.exp(-4.0 * v / 512.0))
    frac = t - np.floor(t)
    assert np.min(np.abs(frac - 0.5)) > 1e-6


def test_int_wsilu_and_gate_round_exactly():
    rng = np.random.default_rng(4)
    h1 = np.concatenate([np.arange(-1100, 1100), rng.integers(-32768, 32768, 3000)])
    h2 = rng.integers(-32768, 32768, h1.size)
    S = ci.sigmoid_table()
    w = ci.int_wsilu(h1)
    g = ci.int_gate(h1, h2)
    for a, b, ww, gg in zip(h1[::7], h2[::7], w[::7], g[::7]):
        a, b = int(a), int(b)
        want_w = round(Fraction(a * int(S[a + 32768]), 512))  # Python rounds halves to even
        assert ww == want_w
        want_g = max(-32768, min(32767, round(Fraction(want_w * b, 512))))
        assert gg == want_g
    assert np.all(np.abs(w) <= np.abs(h1))


def brute_gated_block(z, blk):
    """Nested loops straight from the definition (float64)."""
    C, H, W = z.shape
    out = np.array(z, dtype=np.float64)
    for y in range(H):
        for x in range(W):
            a = np.zeros(C)
            for c in range(C):
                s = blk.dw.b[c]
                for dy in (-1, 0, 1):
                    for dx in (-1, 0, 1):
                        if 0 <= y + dy < H and 0 <= x + dx < W:
                            s += blk.dw.w[c, dy + 1, dx + 1] * z[c, y + dy, x + dx]
                a[c] = s
            h = blk.pw1.w @ a + blk.pw1.b
            g = np.array([h[c] / (1.0 + math.exp(-4.0 * h[c])) * h[C + c] for c in range(C)])
            out[:, y, x] += blk.pw2.w @ g + blk.pw2.b
    return out


def brute_int_gated_block(z, b):
    C, H, W = z.shape
    S = ci.sigmoid_table()

    def rq(num, den):
        return round(Fraction(int(num), int(den)))

    def c16(v):
        return max(-32768, min(32767, v))

    out = np.zeros_like(z)
    for y in range(H):
        for x in range(W):
            a = []
            for c in range(C):
                acc = 512 * int(b.dw.b[c])
                for dy in (-1, 0, 1):
                    for dx in (-1, 0, 1):
                        if 0 <= y + dy < H and 0 <= x + dx < W:
                            acc += int(b.dw.w[c, dy + 1, dx + 1]) * int(z[c, y + dy, x + dx])
                a.append(c16(rq(acc, 8192)))
            h = [c16(rq(512 * int(b.pw1.b[n]) + sum(int(b.pw1.w[n, k]) * a[k] for k in range(C)), 8192))
                 for n in range(2 * C)]
            g = []
            for c in range(C):
                ws = rq(h[c] * int(S[h[c] + 32768]), 512)
                g.append(c16(rq(ws * h[C + c], 512)))
            for n in range(C):
                p = c16(rq(512 * int(b.pw2.b[n]) + sum(int(b.pw2.w[n, k]) * g[k] for k in range(C)), 8192))
                out[n, y, x] = c16(int(z[n, y, x]) + p)
    return out


def gated_params(C=8, ne=1, nd=1):
    flat = synth.make_weights(C, ne, nd, block="gated")
    return oracle.unpack(flat, C, ne, nd, block="gated")


def test_gated_parameter_count_and_shapes():
    for C in (8, 64, 256):
        n = sum(int(np.prod(s)) for _, s, _, _ in synth.param_list(C, 2, 3, "gated"))
        assert n == oracle.params.count(C, 2, 3, "gated")
        assert oracle.params.count(C, 2, 3, "lrelu") - n == 5 * C * C
    p = gated_params(16, 2, 1)
    assert p.block == "gated" and p.enc[0].kind == "gated"
    assert p.enc[0].pw1.w.shape == (32, 16) and p.enc[0].pw2.w.shape == (16, 16)
    with pytest.raises(ValueError):
        oracle.unpack(synth.make_weights(16, 2, 1), 16, 2, 1, block="gated")


def test_gated_block_float_matches_brute_force():
    p = gated_params()
    rng = np.random.default_rng(1)
    z = rng.standard_normal((8, 5, 6))
    np.testing.assert_allclose(cf.dc_block(z, p.enc[0]), brute_gated_block(z, p.enc[0]), rtol=1e-12, atol=1e-12)


def test_gated_block_int_matches_brute_force():
    p = gated_params()
    ip = ci.integerize(p)
    rng = np.random.default_rng(2)
    z = rng.integers(-2048, 2048, (8, 4, 5))
    np.testing.assert_array_equal(ci.dc_block(z, ip.enc[0]), brute_int_gated_block(z, ip.enc[0]))


def torch_gated_block(z, blk):
    C = z.shape[1]
    a = F.conv2d(z, t64(blk.dw.w)[:, None], t64(blk.dw.b), padding=1, groups=C)
    h = F.conv2d(a, t64(blk.pw1.w)[:, :, None, None], t64(blk.pw1.b))
    h1, h2 = torch.chunk(h, 2, dim=1)
    g = F.silu(4.0 * h1) / 4.0 * h2
    return z + F.conv2d(g, t64(blk.pw2.w)[:, :, None, None], t64(blk.pw2.b))


def test_gated_transform_matches_torch_blocks():
    pre = synth.PRESETS["tiny"]
    p = gated_params(pre.channels, pre.n_enc, pre.n_dec)
    x = next(iter(synth.frame_sequence(pre, 1)))
    st = cf.zero_state(p, pre.height, pre.width)
    f = cf.encoder_feature(p, x, st.feat)
    u = F.conv2d(t64(x)[None], t64(p.pe.w.reshape(p.C, 3, 8, 8)), t64(p.pe.b), stride=8)
    z = F.conv2d(torch.cat([u, t64(st.feat)[None]], 1), t64(p.fuse_enc.w)[:, :, None, None], t64(p.fuse_enc.b))
    for blk in p.enc:
        z = torch_gated_block(z, blk)
    np.testing.assert_allclose(f, z[0].numpy(), rtol=1e-10, atol=1e-10)


def test_gated_int_path_tracks_float_and_states_agree():
    pre = synth.PRESETS["tiny"]
    p = gated_params(pre.channels, pre.n_enc, pre.n_dec)
    ip = ci.integerize(p)
    frames = list(synth.frame_sequence(pre, 2))
    # first frame, same zero state: y_i / 512 ~ y_f (integerisation error only)
    yf = cf.analysis(p, frames[0], np.zeros((64, 8, 8)))
    yi = ci.analysis(ip, frames[0], np.zeros((64, 8, 8), dtype=np.int64))
    assert np.max(np.abs(yi / 512 - yf)) < 2e-2
    # the int encoder's state equals the int decoder's, frame after frame
    se = ci.zero_state(ip, 64, 64)
    sd = ci.zero_state(ip, 64, 64)
    for x in frames:
        ri = ci.encode_frame(ip, x, se)
        xhat, sd = ci.decode_frame(ip, ri.q, sd)
        np.testing.assert_array_equal(sd.feat, ri.state.feat)
        np.testing.assert_array_equal(sd.yhat, ri.state.yhat)
        se = ri.state


@pytest.mark.parametrize("name", ["tiny", "wvga"])
def test_gated_activations_stay_in_int16_range(name):
    pre = synth.PRESETS[name]
    p = gated_params(pre.channels, pre.n_enc, pre.n_dec)
    ip = ci.integerize(p)
    st = ci.zero_state(ip, pre.height, pre.width)
    for x in synth.frame_sequence(pre, 2):
        r = ci.encode_frame(ip, x, st)   # raises OverflowError on any int32 overflow
        st = r.state
        assert np.max(np.abs(st.feat)) < 16 * 512


def test_sigmoid_table_compact_form():
    # the integer gated block keeps S in a compact exact form: S[v] - 256 for
    # 0 <= v < 888 (one byte each), S[v] = 512 from 888 on, S[-v] = 512 - S[v]
    S = ci.sigmoid_table()
    v = np.arange(0, 32768)
    pos = S[v + 32768]
    assert np.all(pos[888:] == 512) and pos[887] == 511
    assert np.all((pos[:888] >= 256) & (pos[:888] <= 511))
    np.testing.assert_array_equal(S[32768 - v[1:]], 512 - pos[1:])
    assert S[0] == 0  # v = -32768
