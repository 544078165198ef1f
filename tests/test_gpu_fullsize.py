"""Full-size parity in the configuration bench.py times: 1920x1088 (fp16 and int16)
and 3840x2176 (fp16), C = 256, 8 + 8 blocks, over the whole sequences (32 and
16 frames).

Integer path: the GPU runs the 32-frame 1080p sequence free-running (each frame
coded from its own previous state, as a low-delay encoder and decoder do) and
every frame's q, yhat_t, f_t and xhat must hash to the digests the CPU oracle
wrote for the same sequence (tests/golden/make_hd1080_int_digests.py), and its
bit estimate must equal the oracle's to 1e-5: cross-device consistency of the
integerised model (Sec. 4.5; supplementary "Model Integerization").

fp16 path: the GPU codes whole frames.  On every frame the frame's bit total is
compared with the oracle's rate of the GPU's symbols under the oracle's prior
on the GPU's previous latent, and one sampled region is recomputed by the
teacher-forced oracle (the region rotates over three positions from frame to
frame).  The oracle recomputes sampled regions: every output
of the transform depends only on inputs within a bounded neighbourhood (each 3x3
depthwise conv widens it by one pixel at 1/8 scale; everything else is 1x1, 2x2/s2 or
a pixel shuffle), so the oracle run on a crop of the frame and of the GPU's state
reproduces the full-frame result exactly away from the crop's artificial borders.
Crops touching the real frame border keep that border (zero padding is then the same).
"""
import hashlib
import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import codec_float as cf
from oracle import codec_int as ci
from paper_2502_20762_amd.ncodec import Codec

from parity_util import assert_close_fp16, check_fp16_encode, params_for

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

DEV = "cuda:0"
S = 28        # crop size in latent (1/16) pixels
MARGIN = 10   # latent pixels discarded at crop borders interior to the frame


def geometry(pre):
    H16, W16 = pre.height // 16, pre.width // 16
    # top-left corner, bottom-right corner, an interior crop
    crops = [(0, 0), (H16 - S, W16 - S), (H16 // 3, W16 // 2 - 14)]
    return pre.height, pre.width, pre.channels, pre.n_enc, pre.n_dec, H16, W16, crops


def say(*a):
    print("[gpu-fullsize]", *a, flush=True)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def crop_views(Y0, X0, H16, W16):
    """Slices of the crop inside the full arrays, and of the valid region inside the crop."""
    lo_y = MARGIN if Y0 > 0 else 0
    lo_x = MARGIN if X0 > 0 else 0
    hi_y = S - (MARGIN if Y0 + S < H16 else 0)
    hi_x = S - (MARGIN if X0 + S < W16 else 0)
    full = {k: (slice(f * Y0, f * (Y0 + S)), slice(f * X0, f * (X0 + S))) for k, f in (("l", 1), ("f", 2), ("x", 16))}
    valid = {k: (slice(f * lo_y, f * hi_y), slice(f * lo_x, f * hi_x)) for k, f in (("l", 1), ("f", 2), ("x", 16))}
    return full, valid


def frames(pre):
    return list(synth.frame_sequence(pre, 2))


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hd1080_int_digests.json")


def digest(a):
    return hashlib.sha256(np.ascontiguousarray(np.asarray(a).astype("<i2")).tobytes()).hexdigest()


def test_hd1080_int_free_running_digests():
    g = json.load(open(GOLDEN))
    pre = synth.PRESETS["hd1080_int"]
    assert (g["height"], g["width"], g["channels"], g["n_enc"], g["n_dec"]) == \
        (pre.height, pre.width, pre.channels, pre.n_enc, pre.n_dec)
    assert len(g["frames"]) == pre.n_frames
    H, W, C, NE, ND = pre.height, pre.width, pre.channels, pre.n_enc, pre.n_dec
    flat, _ = params_for(C, NE, ND)
    enc = Codec(H, W, C, NE, ND, "int16", flat, device=DEV)
    dec = Codec(H, W, C, NE, ND, "int16", flat, device=DEV)
    for t, x in enumerate(synth.frame_sequence(pre)):
        ref = g["frames"][t]
        q, bits = enc.encode(torch.from_numpy(x).to(DEV))
        xhat = dec.decode(q)
        f1, y1 = enc.get_state()
        d1, e1 = dec.get_state()
        got = {"q": digest(host(q)), "yhat": digest(host(y1)), "feat": digest(host(f1)), "xhat": digest(host(xhat))}
        say(f"int free-running frame {t}: bits {float(host(bits)):.1f} (oracle {ref['bits']:.1f})")
        assert torch.equal(d1, f1) and torch.equal(e1, y1), f"frame {t}: decoder state differs from encoder state"
        for k, v in got.items():
            assert v == ref[k], f"frame {t}: {k} differs from the oracle's free-running sequence"
        assert abs(float(host(bits)) - ref["bits"]) <= 1e-5 * ref["bits"], (t, float(host(bits)), ref["bits"])


def test_hd1080_int_sampled_bit_exact():
    H, W, C, NE, ND, H16, W16, CROPS = geometry(synth.PRESETS["hd1080_int"])
    flat, p = params_for(C, NE, ND)
    ip = ci.integerize(p)
    enc = Codec(H, W, C, NE, ND, "int16", flat, device=DEV)
    dec = Codec(H, W, C, NE, ND, "int16", flat, device=DEV)
    for t, x in enumerate(frames(synth.PRESETS["hd1080_int"])):
        say("int frame", t)
        f0, y0 = (host(v).astype(np.int64) for v in enc.get_state())
        q, _ = enc.encode(torch.from_numpy(x).to(DEV))
        xhat = host(dec.decode(q))
        f1, y1 = (host(v).astype(np.int64) for v in enc.get_state())
        d1, e1 = (host(v).astype(np.int64) for v in dec.get_state())
        np.testing.assert_array_equal(d1, f1)
        np.testing.assert_array_equal(e1, y1)
        qh = host(q).astype(np.int64)
        for (Y0, X0) in CROPS:
            full, valid = crop_views(Y0, X0, H16, W16)
            say("  crop", (Y0, X0))
            st = ci.State(f0[(slice(None),) + full["f"]], y0[(slice(None),) + full["l"]])
            r = ci.encode_frame(ip, x[(slice(None),) + full["x"]], st)
            xr, _ = ci.decode_frame(ip, r.q, st)
            sl, sf, sx = ((slice(None),) + valid[k] for k in ("l", "f", "x"))
            np.testing.assert_array_equal(qh[(slice(None),) + full["l"]][sl], r.q[sl])
            np.testing.assert_array_equal(y1[(slice(None),) + full["l"]][sl], r.state.yhat[sl])
            np.testing.assert_array_equal(f1[(slice(None),) + full["f"]][sf], r.state.feat[sf])
            np.testing.assert_array_equal(xhat[(slice(None),) + full["x"]][sx], xr[sx])


@pytest.mark.parametrize("preset", ["hd1080", "uhd4k"])
def test_fullsize_fp16_every_frame(preset):
    pre = synth.PRESETS[preset]
    H, W, C, NE, ND, H16, W16, CROPS = geometry(pre)
    flat, p = params_for(C, NE, ND)
    enc = Codec(H, W, C, NE, ND, "fp16", flat, device=DEV)
    dec = Codec(H, W, C, NE, ND, "fp16", flat, device=DEV)
    for t, x in enumerate(synth.frame_sequence(pre)):
        f0, y0 = (host(v).astype(np.float64) for v in enc.get_state())
        q, bits = enc.encode(torch.from_numpy(x).to(DEV))
        xhat = host(dec.decode(q)).astype(np.float64)
        f1, y1 = (host(v).astype(np.float64) for v in enc.get_state())
        d1, e1 = (host(v).astype(np.float64) for v in dec.get_state())
        np.testing.assert_array_equal(d1, f1)
        np.testing.assert_array_equal(e1, y1)
        qh = host(q).astype(np.float64)
        # whole-frame rate: the GPU's symbols under the oracle's prior on the GPU's previous latent
        _, s_ref = cf.prior(p, y0)
        ref_bits = oracle.estimate_bits(qh, oracle.sigma_from_s(s_ref))
        b = float(host(bits))
        say(f"{preset} fp16 frame {t}: bits {b:.1f} (oracle {ref_bits:.1f})")
        assert abs(b - ref_bits) <= 1e-2 * ref_bits, (t, b, ref_bits)
        Y0, X0 = CROPS[t % len(CROPS)]
        full, valid = crop_views(Y0, X0, H16, W16)
        fp = f0[(slice(None),) + full["f"]]
        yp = y0[(slice(None),) + full["l"]]
        sl, sf, sx = ((slice(None),) + valid[k] for k in ("l", "f", "x"))
        f_ref, _ = check_fp16_encode(p, x[(slice(None),) + full["x"]], fp, yp,
                                     qh[(slice(None),) + full["l"]], None,
                                     f1[(slice(None),) + full["f"]], y1[(slice(None),) + full["l"]],
                                     what=f"{preset} fp16 t={t} crop {(Y0, X0)}", valid=(sl, sf))
        assert_close_fp16(xhat[(slice(None),) + full["x"]][sx], cf.reconstruct(p, f_ref)[sx],
                          f"{preset} fp16 t={t} crop {(Y0, X0)} xhat")


def test_hd1080_int_frame_bits_whole_frame():
    # whole-frame rate on the int path, frames 0-2: the GPU's symbols under the
    # oracle's exact integer prior on the GPU's previous latent (sigma from the
    # K1-scaled s, float64) against the GPU's fp32 table-driven rate
    pre = synth.PRESETS["hd1080_int"]
    H, W, C, NE, ND = pre.height, pre.width, pre.channels, pre.n_enc, pre.n_dec
    flat, p = params_for(C, NE, ND)
    ip = ci.integerize(p)
    enc = Codec(H, W, C, NE, ND, "int16", flat, device=DEV)
    for t, x in enumerate(synth.frame_sequence(pre, 3)):
        _, y0 = (host(v).astype(np.int64) for v in enc.get_state())
        q, bits = enc.encode(torch.from_numpy(x).to(DEV))
        _, s = ci.prior(ip, y0)
        ref = oracle.estimate_bits(host(q).astype(np.int64), ci.sigma_int(s))
        b = float(host(bits))
        say(f"int frame {t}: bits {b:.1f} (oracle {ref:.1f})")
        assert abs(b - ref) <= 1e-5 * ref, (t, b, ref)


def test_hd720_both_paths():
    # 1280x720 (Tab. 3d's resolution), C = 256, 8 + 8 blocks: fp16 whole frame
    # teacher-forced (two frames), int path two frames free-running compared on
    # three sampled regions (ragged tiles: 90 x 160 at 1/8, 45 x 80 latent)
    H, W, C, NE, ND = 720, 1280, 256, 8, 8
    flat, p = params_for(C, NE, ND)
    xs = [synth.random_frame(H, W, seed=s) for s in (50, 51)]
    enc = Codec(H, W, C, NE, ND, "fp16", flat, device=DEV)
    dec = Codec(H, W, C, NE, ND, "fp16", flat, device=DEV)
    for t, x in enumerate(xs):
        say("720p fp16 frame", t)
        f0, y0 = (host(v).astype(np.float64) for v in enc.get_state())
        q, bits = enc.encode(torch.from_numpy(x).to(DEV))
        xhat = host(dec.decode(q)).astype(np.float64)
        f1, y1 = (host(v).astype(np.float64) for v in enc.get_state())
        f_ref, _ = check_fp16_encode(p, x, f0, y0, host(q), float(host(bits)), f1, y1, what=f"720p t={t}")
        assert_close_fp16(xhat, cf.reconstruct(p, f_ref), f"720p t={t} xhat")
    ip = ci.integerize(p)
    enc = Codec(H, W, C, NE, ND, "int16", flat, device=DEV)
    dec = Codec(H, W, C, NE, ND, "int16", flat, device=DEV)
    H16, W16 = H // 16, W // 16
    for t, x in enumerate(xs):
        say("720p int frame", t)
        f0, y0 = (host(v).astype(np.int64) for v in enc.get_state())
        q, _ = enc.encode(torch.from_numpy(x).to(DEV))
        xhat = host(dec.decode(q))
        f1, y1 = (host(v).astype(np.int64) for v in enc.get_state())
        qh = host(q).astype(np.int64)
        for (Y0, X0) in [(0, 0), (H16 - S, W16 - S), (H16 // 3, W16 // 2 - 14)]:
            full, valid = crop_views(Y0, X0, H16, W16)
            st = ci.State(f0[(slice(None),) + full["f"]], y0[(slice(None),) + full["l"]])
            r = ci.encode_frame(ip, x[(slice(None),) + full["x"]], st)
            xr, _ = ci.decode_frame(ip, r.q, st)
            sl, sf, sx = ((slice(None),) + valid[k] for k in ("l", "f", "x"))
            np.testing.assert_array_equal(qh[(slice(None),) + full["l"]][sl], r.q[sl])
            np.testing.assert_array_equal(y1[(slice(None),) + full["l"]][sl], r.state.yhat[sl])
            np.testing.assert_array_equal(f1[(slice(None),) + full["f"]][sf], r.state.feat[sf])
            np.testing.assert_array_equal(xhat[(slice(None),) + full["x"]][sx], xr[sx])
