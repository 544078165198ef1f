"""Entropy coding on the GPU against the oracle (oracle/entropy.py), through
the C ABI.

* The standalone coder: for the same symbols and scale indices the GPU
  container is byte-identical to the oracle's, and the GPU decodes the
  oracle's container back to the symbols.
* Coded frames: encode_frame_coded -> decode_frame_coded reproduces the
  symbols and the frame of the plain path; the container size is close to the
  estimated bits.
* Int path: the scale indices equal the oracle's (the int prior is exact), so
  the oracle decodes the GPU's container with its own indices: the paper's
  cross-device consistency, with the CPU oracle as the second device.
* Damaged containers are flagged (status bits) without reads past the
  container.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import codec_int as ci
from oracle import entropy as E
from paper_2502_20762_amd.ncodec import Codec

from parity_util import params_for

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def say(*a):
    print("[gpu-entropy]", *a, flush=True)


def gpu(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def symbols(n, seed, esc_every=0):
    rng = np.random.default_rng(seed)
    sig = np.exp(rng.uniform(np.log(0.05), np.log(400.0), n))
    k = E.scale_index(sig)
    q = np.rint(rng.standard_normal(n) * sig)
    if esc_every:
        q[::esc_every] = rng.integers(-32768, 32768, len(q[::esc_every]))
        q[: min(n, 2)] = [-32768, 32767][: min(n, 2)]
    return np.clip(q, -32768, 32767).astype(np.int16), k.astype(np.uint8)


@pytest.fixture(scope="module")
def coder():
    flat, _ = params_for(128, 1, 1)
    return Codec(256, 256, 128, 1, 1, "fp16", flat, device=DEV)  # 32,768 symbols per frame


@pytest.mark.parametrize("n,esc", [(1, 0), (63, 5), (E.STREAM - 1, 41), (E.STREAM, 0), (E.STREAM + 1, 17),
                                   (20000, 97), (32768, 0)])
def test_rans_container_matches_oracle(coder, n, esc):
    say("standalone coder n =", n, "escape every", esc)
    q, k = symbols(n, seed=n + 7, esc_every=esc)
    want = E.encode(q.astype(np.int64), k.astype(np.int64))
    buf, nb = coder.rans_encode(gpu(q), gpu(k))
    nbytes = int(host(nb))
    got = host(buf)[:nbytes].tobytes()
    assert nbytes == len(want), (nbytes, len(want))
    assert got == want
    # the GPU decodes the oracle's container
    back, st = coder.rans_decode(gpu(np.frombuffer(want, np.uint8).copy()), len(want), gpu(k))
    assert int(host(st)) == 0
    np.testing.assert_array_equal(host(back), q)


def test_damaged_containers_are_flagged(coder):
    q, k = symbols(20000, seed=11, esc_every=50)
    buf, nb = coder.rans_encode(gpu(q), gpu(k))
    nbytes = int(host(nb))
    data = host(buf)[:nbytes].copy()
    say("damaged containers, clean size", nbytes)
    kk = gpu(k)
    _, st = coder.rans_decode(gpu(data), nbytes, kk)
    assert int(host(st)) == 0
    bad = data.copy()
    bad[0] ^= 0xFF  # magic
    _, st = coder.rans_decode(gpu(bad), nbytes, kk)
    assert int(host(st)) & 1
    _, st = coder.rans_decode(gpu(data), nbytes - 100, kk)  # truncated
    assert int(host(st)) & 1
    flip = data.copy()
    flip[nbytes - 300] ^= 0x5A  # inside the last stream's words
    out, st = coder.rans_decode(gpu(flip), nbytes, kk)
    assert int(host(st)) != 0 or not np.array_equal(host(out), q)
    _, st = coder.rans_decode(gpu(data), nbytes, kk)  # the context is fine afterwards
    assert int(host(st)) == 0


@pytest.mark.parametrize("path,H,W,C,ne,nd", [("fp16", 64, 64, 64, 2, 2), ("int16", 64, 64, 64, 2, 2),
                                              ("fp16", 480, 832, 128, 2, 2), ("int16", 480, 832, 128, 2, 2),
                                              ("fp16", 1088, 1920, 256, 8, 8), ("int16", 1088, 1920, 256, 8, 8)])
def test_coded_frames_round_trip(path, H, W, C, ne, nd):
    flat, _ = params_for(C, ne, nd)
    enc = Codec(H, W, C, ne, nd, path, flat, device=DEV)
    dec = Codec(H, W, C, ne, nd, path, flat, device=DEV)
    ref = Codec(H, W, C, ne, nd, path, flat, device=DEV)  # plain decode of the same symbols
    odt = torch.int16 if path == "int16" else torch.float16
    for t in range(3):
        say(path, (H, W, C), "frame", t)
        x = gpu(synth.random_frame(H, W, seed=60 + t))
        q = torch.empty(enc.q_shape, dtype=torch.int16, device=DEV)
        bits = torch.zeros((), dtype=torch.float64, device=DEV)
        buf, nb = enc.encode_coded(x, q_out=q, bits_out=bits)
        nbytes = int(host(nb))
        xo, st = dec.decode_coded(buf, nbytes)
        xr = ref.decode(q, out=torch.empty(enc.frame_shape, dtype=odt, device=DEV))
        assert int(host(st)) == 0
        np.testing.assert_array_equal(host(xo), host(xr), err_msg=f"{path} t={t} frame")
        np.testing.assert_array_equal(host(dec.get_state()[1]), host(enc.get_state()[1]), err_msg=f"{path} t={t} yhat")
        est = float(host(bits)) / 8.0
        ns = -(-q.numel() // E.STREAM)
        # container within the estimate plus table quantisation and the per-stream states
        assert nbytes <= 1.10 * est + 256 * ns + 64, (nbytes, est)
        assert nbytes >= 0.80 * est, (nbytes, est)


def test_int_scale_indices_and_cross_decode_with_oracle():
    H, W, C, ne, nd = 64, 96, 64, 1, 1
    flat, p = params_for(C, ne, nd)
    ip = ci.integerize(p)
    enc = Codec(H, W, C, ne, nd, "int16", flat, device=DEV)
    st = ci.zero_state(ip, H, W)
    for t in range(3):
        say("int cross-decode frame", t)
        x = synth.random_frame(H, W, seed=80 + t)
        # scale indices of this frame from the state, GPU and oracle
        k_gpu = host(enc.scale_indices())
        _, s = ci.prior(ip, st.yhat)
        k_ref = E.scale_index(ci.sigma_int(s))
        np.testing.assert_array_equal(k_gpu, k_ref, err_msg=f"t={t} scale indices")
        r = ci.encode_frame(ip, x, st)
        q = torch.empty(enc.q_shape, dtype=torch.int16, device=DEV)
        buf, nb = enc.encode_coded(gpu(x), q_out=q)
        nbytes = int(host(nb))
        data = host(buf)[:nbytes].tobytes()
        np.testing.assert_array_equal(host(q), r.q)
        assert data == E.encode(r.q, k_ref)
        q_or, ok = E.decode(data, k_ref)
        assert ok
        np.testing.assert_array_equal(q_or.reshape(r.q.shape), r.q)
        st = r.state


@pytest.mark.parametrize("path", ["fp16", "int16"])
def test_coded_round_trip_with_gated_blocks_and_modules(path):
    # the coder takes the symbols and scale indices of any model form
    H, W, C, ne, nd = 112, 208, 128, 1, 1
    kw = dict(block="gated", n_fe_blocks=1, n_rg_blocks=1, qp_banks=True)
    flat = synth.make_weights(C, ne, nd, block="gated", n_fe=1, n_rg=1, banks=True)
    enc, dec, ref = (Codec(H, W, C, ne, nd, path, flat, device=DEV, **kw) for _ in range(3))
    odt = torch.int16 if path == "int16" else torch.float16
    for t, qp in enumerate([5, 5, 50]):
        say("coded gated + modules", path, "frame", t, "qp", qp)
        for c in (enc, dec, ref):
            c.set_qp(qp)
        x = gpu(synth.random_frame(H, W, seed=70 + t))
        q = torch.empty(enc.q_shape, dtype=torch.int16, device=DEV)
        buf, nb = enc.encode_coded(x, q_out=q)
        xo, st = dec.decode_coded(buf, int(host(nb)))
        xr = ref.decode(q, out=torch.empty(enc.frame_shape, dtype=odt, device=DEV))
        assert int(host(st)) == 0
        np.testing.assert_array_equal(host(xo), host(xr))
        np.testing.assert_array_equal(host(dec.get_state()[0]), host(enc.get_state()[0]))


@pytest.mark.parametrize("path", ["fp16", "int16"])
def test_parallel_coding_matches_serial(path):
    # Fig. 6 / supplementary "Parallel Coding": the coder on a second stream
    # beside the decoder part of the encode, the feature extractor beside the
    # symbol decoding; containers, symbols, frames and states equal the serial
    # order bit for bit
    H, W, C, ne, nd = 112, 208, 128, 2, 2
    kw = dict(n_fe_blocks=2, n_rg_blocks=1)
    flat = synth.make_weights(C, ne, nd, n_fe=2, n_rg=1)
    se, sd, pe, pd = (Codec(H, W, C, ne, nd, path, flat, device=DEV, **kw) for _ in range(4))
    pe.parallel_coding(True)
    pd.parallel_coding(True)
    for t in range(3):
        say("parallel coding", path, "frame", t)
        x = gpu(synth.random_frame(H, W, seed=90 + t))
        qs = torch.empty(se.q_shape, dtype=torch.int16, device=DEV)
        qp = torch.empty(se.q_shape, dtype=torch.int16, device=DEV)
        bs, ns = se.encode_coded(x, q_out=qs)
        bp, npb = pe.encode_coded(x, q_out=qp)
        n1, n2 = int(host(ns)), int(host(npb))
        assert n1 == n2
        np.testing.assert_array_equal(host(bs)[:n1], host(bp)[:n2])
        np.testing.assert_array_equal(host(qs), host(qp))
        xs, st1 = sd.decode_coded(bs, n1)
        xp, st2 = pd.decode_coded(bp, n2)
        assert int(host(st1)) == 0 and int(host(st2)) == 0
        np.testing.assert_array_equal(host(xs), host(xp))
        for a, b in ((se, pe), (sd, pd), (pe, pd)):
            fa, ya = a.get_state()
            fb, yb = b.get_state()
            assert torch.equal(fa, fb) and torch.equal(ya, yb)
