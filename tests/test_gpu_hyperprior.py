"""GPU parity of the two-step entropy model with the hyper latent z (Sec. 4.4;
supplementary "Entropy model", "Parallel Coding") through the C ABI.

int path: free-running, bit-exact against the oracle on every symbol (y and z),
the latent state, the context and the reconstruction, and the rate to 1e-5.
fp16 path: teacher-forced step by step (the oracle takes the GPU's previous
state, then the GPU's z symbols for the hyper parameters, then the GPU's
y^1 symbols for the second step): every symbol equal outside the fp16 rounding
band and off by at most one inside it; latent, context and reconstruction
within 2e-2 max(1, |ref|); rate within 1e-2.
Coded: the three containers (z, y^1, y^2) decode to the same frames and states
as the plain path, and on the int path the oracle's coder produces the GPU's
containers byte for byte from the oracle's own scale indices.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import codec_float as cf
from oracle import codec_int as ci
from oracle import entropy as E
from oracle import hyperprior as hp
from oracle.ops import conv2x2s2
from paper_2502_20762_amd.ncodec import Codec, _capacity

from parity_util import FP16_TOL, assert_close_fp16

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def say(*a):
    print("[gpu-hyper]", *a, flush=True)


def gpu(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def split_q(q, C, H, W):
    ny = C * (H // 16) * (W // 16)
    return q[:ny].reshape(C, H // 16, W // 16), q[ny:].reshape(64, H // 32, W // 32)


def params(C, ne, nd):
    flat = synth.make_weights(C, ne, nd, hyper=True)
    return flat, oracle.unpack(flat, C, ne, nd, hyper=True)


def band(v, tol=FP16_TOL):
    frac = v - np.floor(v)
    return np.abs(frac - 0.5) <= tol * np.maximum(1.0, np.abs(v))


def check_q(q, v, what):
    """q = round(v) outside the rounding band, within one inside it."""
    ref = np.rint(v)
    b = band(v)
    assert not ((q != ref) & ~b).any(), f"{what}: {int(((q != ref) & ~b).sum())} symbols differ outside the band"
    assert not (np.abs(q - ref) > 1).any(), f"{what}: a symbol is off by more than one"
    assert np.mean(q == ref) > 0.99, what


@pytest.mark.parametrize("H,W,C,ne,nd", [(64, 96, 128, 2, 2), (96, 160, 256, 1, 2)])
def test_hyperprior_int_bit_exact(H, W, C, ne, nd):
    flat, p = params(C, ne, nd)
    ip, ih = ci.integerize(p), hp.integerize_hyper(p)
    enc = Codec(H, W, C, ne, nd, "int16", flat, device=DEV, hyperprior=True)
    dec = Codec(H, W, C, ne, nd, "int16", flat, device=DEV, hyperprior=True)
    st = ci.zero_state(ip, H, W)
    for t in range(3):
        say("int", (H, W, C), "frame", t)
        x = synth.random_frame(H, W, seed=100 + t)
        r = hp.encode_frame_int(p, ip, ih, x, st)
        q, bits = enc.encode(gpu(x))
        qy, qz = split_q(host(q), C, H, W)
        np.testing.assert_array_equal(qz, r.sym.qz, err_msg=f"t={t} z symbols")
        np.testing.assert_array_equal(qy, r.sym.y(), err_msg=f"t={t} y symbols")
        f, y = (host(v).astype(np.int64) for v in enc.get_state())
        np.testing.assert_array_equal(f, r.state.feat, err_msg=f"t={t} f_t")
        np.testing.assert_array_equal(y, r.state.yhat, err_msg=f"t={t} yhat")
        assert abs(float(host(bits)) - r.bits) <= 1e-5 * r.bits, (float(host(bits)), r.bits)
        xr, _ = hp.decode_frame_int(ip, ih, r.sym, st)
        np.testing.assert_array_equal(host(dec.decode(q)), xr, err_msg=f"t={t} xhat")
        df, dy = dec.get_state()
        assert torch.equal(df, enc.get_state()[0]) and torch.equal(dy, enc.get_state()[1])
        st = r.state


def test_hyperprior_fp16_teacher_forced():
    H, W, C, ne, nd = 64, 96, 128, 2, 2
    flat, p = params(C, ne, nd)
    enc = Codec(H, W, C, ne, nd, "fp16", flat, device=DEV, hyperprior=True)
    dec = Codec(H, W, C, ne, nd, "fp16", flat, device=DEV, hyperprior=True)
    H2 = C // 2
    for t in range(3):
        say("fp16 frame", t)
        x = synth.random_frame(H, W, seed=110 + t)
        f0, y0 = (host(v).astype(np.float64) for v in enc.get_state())
        q, bits = enc.encode(gpu(x))
        qy, qz = (v.astype(np.float64) for v in split_q(host(q), C, H, W))
        f1, y1 = (host(v).astype(np.float64) for v in enc.get_state())
        y = cf.analysis(p, x, f0)
        check_q(qz, conv2x2s2(y, p.hyper.zana.w, p.hyper.zana.b), f"t={t} z")
        mu_h, s_h = hp.hyper_params_float(p, qz)
        mu_t, s_t = cf.prior(p, y0)
        mu, s = mu_t + mu_h, s_t + s_h
        check_q(qy[:H2], y[:H2] - mu[:H2], f"t={t} y^1")
        yhat1 = qy[:H2] + mu[:H2]
        dmu, ds = hp.step2_float(p, yhat1)
        check_q(qy[H2:], y[H2:] - (mu[H2:] + dmu), f"t={t} y^2")
        yhat = np.concatenate([yhat1, qy[H2:] + mu[H2:] + dmu])
        assert_close_fp16(y1, yhat, f"t={t} yhat")
        f_ref = cf.decoder_feature(p, yhat, f0)
        assert_close_fp16(f1, f_ref, f"t={t} f_t")
        sym = hp.Symbols(qz, qy[:H2], qy[H2:])
        rb = sum(hp.rates(p, sym, oracle.sigma_from_s(s[:H2]), oracle.sigma_from_s(s[H2:] + ds)))
        assert abs(float(host(bits)) - rb) <= 1e-2 * rb, (float(host(bits)), rb)
        xh = host(dec.decode(q)).astype(np.float64)
        df, dy = dec.get_state()
        assert torch.equal(df, enc.get_state()[0]) and torch.equal(dy, enc.get_state()[1])
        assert_close_fp16(xh, cf.reconstruct(p, f_ref), f"t={t} xhat")


@pytest.mark.parametrize("path", ["fp16", "int16"])
def test_hyperprior_coded_round_trip(path):
    H, W, C, ne, nd = 96, 160, 128, 1, 1
    flat, p = params(C, ne, nd)
    enc, dec, ref = (Codec(H, W, C, ne, nd, path, flat, device=DEV, hyperprior=True) for _ in range(3))
    dec.parallel_coding(path == "int16")  # both orders of the decoder
    if path == "int16":
        ip, ih = ci.integerize(p), hp.integerize_hyper(p)
        st = ci.zero_state(ip, H, W)
    odt = torch.int16 if path == "int16" else torch.float16
    for t in range(3):
        say("coded", path, "frame", t)
        x = synth.random_frame(H, W, seed=120 + t)
        q = torch.empty(enc.q_shape, dtype=torch.int16, device=DEV)
        buf, nb = enc.encode_coded(gpu(x), q_out=q)
        xo, status = dec.decode_coded(buf, buf.numel())
        xr = ref.decode(q, out=torch.empty(enc.frame_shape, dtype=odt, device=DEV))
        assert (host(status) == 0).all()
        np.testing.assert_array_equal(host(xo), host(xr))
        for a, b in zip(dec.get_state(), enc.get_state()):
            assert torch.equal(a, b)
        if path == "int16":
            r = hp.encode_frame_int(p, ip, ih, x, st)
            qy, qz = split_q(host(q), C, H, W)
            np.testing.assert_array_equal(qz, r.sym.qz)
            np.testing.assert_array_equal(qy, r.sym.y())
            data, lens = host(buf), host(nb)
            nz, nh = qz.size, qy.size // 2
            off = [0, _capacity(nz), _capacity(nz) + _capacity(nh)]
            kz = np.broadcast_to(E.scale_index(hp.z_sigma(p))[:, None, None], qz.shape)
            ks = [kz, E.scale_index(r.sigma1), E.scale_index(r.sigma2)]
            for i, (sq, k) in enumerate(zip([r.sym.qz, r.sym.q1, r.sym.q2], ks)):
                got = data[off[i]:off[i] + int(lens[i])].tobytes()
                assert got == E.encode(sq, k), f"t={t} container {i}"
            st = r.state


def test_hyperprior_rate_point_selects_nearest_z_module():
    H, W, C = 64, 96, 128
    flat, p = params(C, 1, 1)
    x = gpu(synth.random_frame(H, W, seed=130))
    out = []
    for qp in (0.0, 20.4, 20.6):
        c = Codec(H, W, C, 1, 1, "int16", flat, device=DEV, hyperprior=True)
        if qp:
            c.set_rate(qp)
        _, bits = c.encode(x)
        out.append(float(host(bits)))
    ip, ih = ci.integerize(p), hp.integerize_hyper(p)
    xs = host(x)
    for qp, b in zip((0.0, 20.4, 20.6), out):
        r = hp.encode_frame_int(p, ip, ih, xs, ci.zero_state(ip, H, W), qp=qp)
        assert abs(b - r.bits) <= 1e-5 * r.bits, (qp, b, r.bits)
    assert out[0] != out[1] != out[2]


def windows(h16, w16):
    """Even-aligned windows of the 1/16 grid: first, middle and the last
    (ragged) corner; every step of the entropy model is local to a 2 x 2 cell."""
    return [(0, 0, 8, 8), (h16 // 2 & ~1, w16 // 2 & ~1, 10, 12), (h16 - 6, w16 - 8, 6, 8)]


@pytest.mark.parametrize("path", ["int16", "fp16"])
def test_hyperprior_hd1080_windows(path):
    """The benchmarked 1080p configuration (C = 256, 8 + 8 blocks) with the
    two-step model: on sampled windows the oracle recomputes the latent from the
    GPU's symbols and previous latent (hyper-synthesis, step 1, y^1, step 2,
    y^2), bit-exact on the int path; the decoder, fed the three containers,
    reproduces the encoder's state bit for bit."""
    H, W, C, ne, nd = 1088, 1920, 256, 8, 8
    flat, p = params(C, ne, nd)
    enc, dec = (Codec(H, W, C, ne, nd, path, flat, device=DEV, hyperprior=True) for _ in range(2))
    ip, ih = (ci.integerize(p), hp.integerize_hyper(p)) if path == "int16" else (None, None)
    frames = synth.frame_sequence("hd1080", 3)
    for t, x in enumerate(frames):
        say("hd1080", path, "frame", t)
        _, y0 = (host(v).astype(np.int64 if ip else np.float64) for v in enc.get_state())
        q = torch.empty(enc.q_shape, dtype=torch.int16, device=DEV)
        buf, nb = enc.encode_coded(gpu(x.astype(np.float16)), q_out=q)
        _, status = dec.decode_coded(buf, buf.numel())
        assert (host(status) == 0).all()
        for a, b in zip(dec.get_state(), enc.get_state()):
            assert torch.equal(a, b)
        y1 = host(enc.get_state()[1]).astype(np.float64)
        qy, qz = split_q(host(q), C, H, W)
        for (Y, X, h, w) in windows(H // 16, W // 16):
            sym = hp.Symbols(qz[:, Y // 2:(Y + h) // 2, X // 2:(X + w) // 2],
                             qy[:C // 2, Y:Y + h, X:X + w], qy[C // 2:, Y:Y + h, X:X + w])
            if ip is not None:
                ref, _, _ = hp.latent_from_symbols_int(ip, ih, sym, y0[:, Y:Y + h, X:X + w])
                np.testing.assert_array_equal(y1[:, Y:Y + h, X:X + w], ref, err_msg=f"t={t} window {(Y, X)}")
            else:
                ref, _, _ = hp.latent_from_symbols_float(p, sym, y0[:, Y:Y + h, X:X + w])
                assert_close_fp16(y1[:, Y:Y + h, X:X + w], ref, f"t={t} window {(Y, X)}")
