"""Whole-transform pins for the oracle.

The float transform is checked against an independent re-implementation built
from different library primitives (strided / grouped / transposed convolutions
of torch.nn.functional in float64 on the CPU); the integer transform against
its own invariants (encoder state == decoder state, determinism) and against
the float transform it approximates.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth
from oracle import codec_float as cf
from oracle import codec_int as ci


def t64(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))


def torch_block(z, blk):
    C = z.shape[1]
    a = F.conv2d(z, t64(blk.dw.w)[:, None], t64(blk.dw.b), padding=1, groups=C)
    h = F.conv2d(a, t64(blk.pw1.w)[:, :, None, None], t64(blk.pw1.b))
    return z + F.conv2d(F.leaky_relu(h, 0.1), t64(blk.pw2.w)[:, :, None, None], t64(blk.pw2.b))


def torch_transform(p, x, f_prev, yhat_prev):
    """Float transform from strided/transposed convolutions (no pixel (un)shuffle)."""
    C = p.C
    x = t64(x)[None]
    e = F.conv2d(x, t64(p.pe.w.reshape(C, 3, 8, 8)), t64(p.pe.b), stride=8)
    z = F.conv2d(torch.cat([e, t64(f_prev)[None]], 1), t64(p.fuse_enc.w)[:, :, None, None], t64(p.fuse_enc.b))
    for blk in p.enc:
        z = torch_block(z, blk)
    y = F.conv2d(z, t64(p.down.w), t64(p.down.b), stride=2)
    ms = F.conv2d(t64(yhat_prev)[None], t64(p.head.w)[:, :, None, None], t64(p.head.b))
    mu = ms[:, :C]
    q = torch.round(y - mu)
    yhat = q + mu
    wt = t64(p.up.w.reshape(C, 2, 2, C).transpose(3, 0, 1, 2))
    d = F.conv_transpose2d(yhat, wt, None, stride=2)
    bias = t64(p.up.b.reshape(C, 2, 2))
    d = d + bias.repeat(1, d.shape[2] // 2, d.shape[3] // 2)[None]
    z = F.conv2d(torch.cat([d, t64(f_prev)[None]], 1), t64(p.fuse_dec.w)[:, :, None, None], t64(p.fuse_dec.b))
    for blk in p.dec:
        z = torch_block(z, blk)
    wr = t64(p.rec.w.reshape(3, 8, 8, C).transpose(3, 0, 1, 2))
    r = F.conv_transpose2d(z, wr, None, stride=8)
    r = r + t64(p.rec.b.reshape(3, 8, 8)).repeat(1, r.shape[2] // 8, r.shape[3] // 8)[None]
    xhat = torch.clamp(r, 0, 1)
    return y[0].numpy(), mu[0].numpy(), q[0].numpy(), z[0].numpy(), xhat[0].numpy()


def tiny():
    pre = synth.PRESETS["tiny"]
    flat = synth.make_weights(pre.channels, pre.n_enc, pre.n_dec)
    return pre, oracle.unpack(flat, pre.channels, pre.n_enc, pre.n_dec)


def test_parameter_count():
    # hand count for C = 64, 2 + 2 blocks
    assert oracle.params.count(64, 2, 2) == 151616
    for C, ne, nd in [(64, 2, 2), (128, 6, 6), (256, 8, 8)]:
        n = sum(int(np.prod(s)) for _, s, _, _ in synth.param_list(C, ne, nd))
        assert n == oracle.params.count(C, ne, nd)


def test_weights_are_fp16_representable_and_seeded():
    w = synth.make_weights(64, 2, 2)
    np.testing.assert_array_equal(w, w.astype(np.float16).astype(np.float32))
    np.testing.assert_array_equal(w, synth.make_weights(64, 2, 2))


def test_float_transform_matches_torch_reimplementation():
    pre, p = tiny()
    st = cf.zero_state(p, pre.height, pre.width)
    for x in synth.frame_sequence(pre):
        r = cf.encode_frame(p, x, st)
        y, mu, q, f, _ = torch_transform(p, x, st.feat, st.yhat)
        np.testing.assert_allclose(r.y, y, atol=1e-11)
        np.testing.assert_allclose(r.mu, mu, atol=1e-11)
        np.testing.assert_array_equal(r.q, q)
        np.testing.assert_allclose(r.state.feat, f, atol=1e-10)
        xhat, sd = cf.decode_frame(p, r.q, st)
        _, _, _, _, xr = torch_transform(p, x, st.feat, st.yhat)
        np.testing.assert_allclose(xhat, xr, atol=1e-10)
        np.testing.assert_array_equal(sd.feat, r.state.feat)
        st = r.state


def test_shapes_of_outputs():
    pre, p = tiny()
    st = cf.zero_state(p, 64, 64)
    x = next(synth.frame_sequence(pre))
    r = cf.encode_frame(p, x, st)
    assert r.q.shape == (64, 4, 4) and r.state.feat.shape == (64, 8, 8)
    xhat, _ = cf.decode_frame(p, r.q, st)
    assert xhat.shape == (3, 64, 64) and xhat.min() >= 0 and xhat.max() <= 1


def test_int_encoder_and_decoder_states_agree_and_are_deterministic():
    pre, p = tiny()
    ip = ci.integerize(p)
    se = ci.zero_state(ip, 64, 64)
    sd = ci.zero_state(ip, 64, 64)
    for x in synth.frame_sequence(pre, 3):
        r1 = ci.encode_frame(ip, x, se)
        r2 = ci.encode_frame(ip, x, se)
        np.testing.assert_array_equal(r1.q, r2.q)
        xhat, sd = ci.decode_frame(ip, r1.q, sd)
        np.testing.assert_array_equal(sd.feat, r1.state.feat)
        np.testing.assert_array_equal(sd.yhat, r1.state.yhat)
        assert xhat.dtype == np.int64 and xhat.min() >= 0 and xhat.max() <= 512
        se = r1.state


def test_decoder_state_desync_changes_output():
    # resetting only the decoder mid-stream must change the reconstruction (state matters)
    pre, p = tiny()
    ip = ci.integerize(p)
    se = ci.zero_state(ip, 64, 64)
    frames = list(synth.frame_sequence(pre, 2))
    r0 = ci.encode_frame(ip, frames[0], se)
    r1 = ci.encode_frame(ip, frames[1], r0.state)
    _, sd0 = ci.decode_frame(ip, r0.q, se)
    good, _ = ci.decode_frame(ip, r1.q, sd0)
    bad, _ = ci.decode_frame(ip, r1.q, ci.zero_state(ip, 64, 64))
    assert not np.array_equal(good, bad)


def test_int_transform_approximates_float_transform():
    # first frame, same zero state: y_i / 512 ~ y_f (integerisation error only)
    pre, p = tiny()
    ip = ci.integerize(p)
    x = next(synth.frame_sequence(pre))
    yf = cf.analysis(p, x, np.zeros((64, 8, 8)))
    yi = ci.analysis(ip, x, np.zeros((64, 8, 8), dtype=np.int64))
    assert np.max(np.abs(yi / 512 - yf)) < 2e-2
    # with the same symbols, reconstructions agree to the integer grid
    mu_f, _ = cf.prior(p, np.zeros((64, 4, 4)))
    q = np.rint(yf - mu_f)
    xf, _ = cf.decode_frame(p, q, cf.zero_state(p, 64, 64))
    xi, _ = ci.decode_frame(ip, q.astype(np.int64), ci.zero_state(ip, 64, 64))
    assert np.max(np.abs(xi / 512 - xf)) < 2e-2


@pytest.mark.parametrize("name", ["tiny", "wvga"])
def test_activations_stay_in_int16_range(name):
    pre = synth.PRESETS[name]
    p = oracle.unpack(synth.make_weights(pre.channels, pre.n_enc, pre.n_dec), pre.channels, pre.n_enc, pre.n_dec)
    ip = ci.integerize(p)
    st = ci.zero_state(ip, pre.height, pre.width)
    for x in synth.frame_sequence(pre, 2):
        r = ci.encode_frame(ip, x, st)   # raises OverflowError on any int32 overflow
        st = r.state
        assert np.max(np.abs(st.feat)) < 16 * 512


def test_crop_locality_used_by_full_size_sampling():
    # The full-size GPU tests compare crops: with 8 + 8 blocks every output more than
    # 10 latent pixels from a crop border depends only on inputs inside the crop.
    import test_gpu_fullsize as fs
    C, ne, nd = 64, 8, 8
    Hf, Wf = 32 * 16, 48 * 16
    p = oracle.unpack(synth.make_weights(C, ne, nd), C, ne, nd)
    ip = ci.integerize(p)
    rng = np.random.default_rng(3)
    x = rng.uniform(0, 1, (3, Hf, Wf)).astype(np.float16)
    st = ci.State(rng.integers(-2000, 2000, (C, Hf // 8, Wf // 8)), rng.integers(-2000, 2000, (C, Hf // 16, Wf // 16)))
    r = ci.encode_frame(ip, x, st)
    xr, _ = ci.decode_frame(ip, r.q, st)
    S, M = fs.S, fs.MARGIN
    for (Y0, X0) in [(0, 0), (32 - S, 48 - S), (2, 11)]:
        sub = ci.State(st.feat[:, 2 * Y0:2 * (Y0 + S), 2 * X0:2 * (X0 + S)], st.yhat[:, Y0:Y0 + S, X0:X0 + S])
        rc = ci.encode_frame(ip, x[:, 16 * Y0:16 * (Y0 + S), 16 * X0:16 * (X0 + S)], sub)
        xc, _ = ci.decode_frame(ip, rc.q, sub)
        ly, lx = (M if Y0 > 0 else 0), (M if X0 > 0 else 0)
        hy, hx = S - (M if Y0 + S < 32 else 0), S - (M if X0 + S < 48 else 0)
        np.testing.assert_array_equal(rc.q[:, ly:hy, lx:hx], r.q[:, Y0 + ly:Y0 + hy, X0 + lx:X0 + hx])
        np.testing.assert_array_equal(rc.state.feat[:, 2 * ly:2 * hy, 2 * lx:2 * hx],
                                      r.state.feat[:, 2 * (Y0 + ly):2 * (Y0 + hy), 2 * (X0 + lx):2 * (X0 + hx)])
        np.testing.assert_array_equal(xc[:, 16 * ly:16 * hy, 16 * lx:16 * hx],
                                      xr[:, 16 * (Y0 + ly):16 * (Y0 + hy), 16 * (X0 + lx):16 * (X0 + hx)])
