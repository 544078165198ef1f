"""GPU parity of the conditional-coding modules (Fig. 4; Sec. 4.3, 4.4) through
the C ABI: feature extractor (N_f DC blocks giving the temporal context),
reconstruction generation (N_r DC blocks before the reconstruction conv) and
the qp vector banks folded into the adjacent convolutions (ncodec_set_qp).

fp16 teacher-forced within 2e-2 max(1, |oracle|), int path bit-exact
free-running; the rate point changes mid-sequence on encoder and decoder
together; both block forms.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import codec_float as cf
from oracle import codec_int as ci
from oracle.params import fold_qp
from paper_2502_20762_amd.ncodec import Codec, NcodecError

from parity_util import assert_close_fp16, check_fp16_encode

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def say(*a):
    print("[gpu-modules]", *a, flush=True)


def gpu(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def setup(H, W, C, ne, nd, nfe, nrg, path, block="lrelu"):
    flat = synth.make_weights(C, ne, nd, block=block, n_fe=nfe, n_rg=nrg, banks=True)
    p = oracle.unpack(flat, C, ne, nd, block=block, n_fe=nfe, n_rg=nrg, banks=True)
    kw = dict(device=DEV, block=block, n_fe_blocks=nfe, n_rg_blocks=nrg, qp_banks=True)
    return p, Codec(H, W, C, ne, nd, path, flat, **kw), Codec(H, W, C, ne, nd, path, flat, **kw)


QPS = [0, 0, 40, 63]  # rate point of each frame


@pytest.mark.parametrize("block", ["lrelu", "gated"])
def test_modules_fp16(block):
    H, W, C, ne, nd, nfe, nrg = 64, 96, 64, 2, 2, 2, 1
    p, enc, dec = setup(H, W, C, ne, nd, nfe, nrg, "fp16", block)
    for t, qp in enumerate(QPS):
        say("fp16", block, "frame", t, "qp", qp)
        enc.set_qp(qp)
        dec.set_qp(qp)
        pq = fold_qp(p, qp)
        x = synth.random_frame(H, W, seed=30 + t)
        f0, y0 = (host(v).astype(np.float64) for v in enc.get_state())
        q, bits = enc.encode(gpu(x))
        f1, y1 = (host(v).astype(np.float64) for v in enc.get_state())
        f_ref, _ = check_fp16_encode(pq, x, f0, y0, host(q), float(host(bits)), f1, y1, f"modules fp16 t={t}")
        xhat = host(dec.decode(q)).astype(np.float64)
        d1, e1 = (host(v).astype(np.float64) for v in dec.get_state())
        np.testing.assert_array_equal(d1, f1)
        np.testing.assert_array_equal(e1, y1)
        assert_close_fp16(xhat, cf.reconstruct(pq, f_ref), f"modules fp16 t={t} xhat")


@pytest.mark.parametrize("H,W,C,ne,nd,nfe,nrg,block", [
    (64, 96, 64, 2, 2, 2, 1, "lrelu"),
    (64, 96, 64, 1, 1, 1, 2, "gated"),
    (112, 208, 256, 1, 1, 1, 1, "lrelu"),   # ragged tiles at C = 256
    (480, 832, 128, 2, 2, 2, 2, "lrelu"),
])
def test_modules_int_bit_exact(H, W, C, ne, nd, nfe, nrg, block):
    p, enc, dec = setup(H, W, C, ne, nd, nfe, nrg, "int16", block)
    st = None
    for t, qp in enumerate(QPS[:3] if H < 400 else [0, 50]):
        say("int", (H, W, C, ne, nd, nfe, nrg, block), "frame", t, "qp", qp)
        enc.set_qp(qp)
        dec.set_qp(qp)
        ip = ci.integerize(fold_qp(p, qp))
        if st is None:
            st = ci.zero_state(ip, H, W)
        x = synth.random_frame(H, W, seed=40 + t)
        r = ci.encode_frame(ip, x, st)
        q, bits = enc.encode(gpu(x))
        np.testing.assert_array_equal(host(q), r.q, err_msg=f"t={t} q")
        f, y = (host(v).astype(np.int64) for v in enc.get_state())
        np.testing.assert_array_equal(f, r.state.feat, err_msg=f"t={t} f_t")
        np.testing.assert_array_equal(y, r.state.yhat, err_msg=f"t={t} yhat")
        assert abs(float(host(bits)) - r.bits) <= 1e-5 * abs(r.bits)
        xr, _ = ci.decode_frame(ip, r.q, st)
        np.testing.assert_array_equal(host(dec.decode(q)), xr, err_msg=f"t={t} xhat")
        st = r.state


def test_set_qp_errors_and_bits_fall_with_qp():
    H, W, C = 64, 64, 64
    p, enc, _ = setup(H, W, C, 1, 1, 1, 0, "fp16")
    with pytest.raises(NcodecError):
        enc.set_qp(64)
    with pytest.raises(NcodecError):
        enc.set_qp(-1)
    plain = Codec(H, W, C, 1, 1, "fp16", synth.make_weights(C, 1, 1), device=DEV)
    with pytest.raises(NcodecError):
        plain.set_qp(3)
    x = gpu(synth.random_frame(H, W, seed=9))
    bits = []
    for qp in (0, 32, 63):
        enc.reset()
        enc.set_qp(qp)
        _, b = enc.encode(x)
        bits.append(float(host(b)))
    say("bits at qp 0, 32, 63:", bits)
    assert bits[0] > bits[1] > bits[2]


@pytest.mark.parametrize("path", ["int16", "fp16"])
def test_interpolated_rates_match_the_oracle(path):
    # rates between the learned points: linearly interpolated bank vectors
    H, W, C, ne, nd, nfe, nrg = 64, 96, 64, 1, 1, 1, 1
    p, enc, dec = setup(H, W, C, ne, nd, nfe, nrg, path)
    rates = [12.5, 12.5, 40.25, 62.75, 63.0]
    st = None
    for t, qp in enumerate(rates):
        say("interpolated rate", path, "frame", t, "qp", qp)
        enc.set_rate(qp)
        dec.set_rate(qp)
        x = synth.random_frame(H, W, seed=50 + t)
        if path == "int16":
            ip = ci.integerize(fold_qp(p, qp))
            if st is None:
                st = ci.zero_state(ip, H, W)
            r = ci.encode_frame(ip, x, st)
            q, bits = enc.encode(gpu(x))
            np.testing.assert_array_equal(host(q), r.q, err_msg=f"qp={qp} q")
            f, y = (host(v).astype(np.int64) for v in enc.get_state())
            np.testing.assert_array_equal(f, r.state.feat, err_msg=f"qp={qp} f_t")
            np.testing.assert_array_equal(y, r.state.yhat, err_msg=f"qp={qp} yhat")
            xr, _ = ci.decode_frame(ip, r.q, st)
            np.testing.assert_array_equal(host(dec.decode(q)), xr, err_msg=f"qp={qp} xhat")
            st = r.state
        else:
            pq = fold_qp(p, qp)
            f0, y0 = (host(v).astype(np.float64) for v in enc.get_state())
            q, bits = enc.encode(gpu(x))
            f1, y1 = (host(v).astype(np.float64) for v in enc.get_state())
            f_ref, _ = check_fp16_encode(pq, x, f0, y0, host(q), float(host(bits)), f1, y1, f"rate {qp}")
            xhat = host(dec.decode(q)).astype(np.float64)
            assert_close_fp16(xhat, cf.reconstruct(pq, f_ref), f"rate {qp} xhat")
    for bad in (-0.5, 63.01, float("nan")):
        with pytest.raises(NcodecError):
            enc.set_rate(bad)
