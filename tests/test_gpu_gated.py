"""GPU parity of the gated DC-block form (Supp. B.1: WSiLU and Chunk; the int
path's sigmoid table of Sec. 4.5) against the oracle, through the C ABI.

Same rules as the LeakyReLU block: fp16 teacher-forced within
2e-2 max(1, |oracle|), int path bit-exact free-running, at shapes from one
latent pixel to several ragged tiles, 832x480 with 6 + 6 blocks, and sampled
crops of a 1080p int frame with 8 + 8 blocks.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import codec_int as ci
from paper_2502_20762_amd.ncodec import Codec

from parity_util import params_for
from test_gpu_parity import run_fp16_sequence, run_int_sequence
from test_gpu_fullsize import crop_views, geometry

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def say(*a):
    print("[gpu-gated]", *a, flush=True)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def test_gated_tiny_fp16():
    run_fp16_sequence(64, 64, 64, 2, 2, list(synth.frame_sequence("tiny", 3)), "gated tiny fp16", block="gated")


def test_gated_tiny_int_bit_exact():
    run_int_sequence(64, 64, 64, 2, 2, list(synth.frame_sequence("tiny_int", 3)), "gated tiny int", block="gated")


EDGE = [(16, 16, 64, 1, 1), (48, 80, 128, 1, 2), (112, 208, 256, 2, 1)]


@pytest.mark.parametrize("H,W,C,ne,nd", EDGE)
def test_gated_edge_shapes_fp16(H, W, C, ne, nd):
    frames = [synth.random_frame(H, W, seed=s) for s in (20, 21)]
    run_fp16_sequence(H, W, C, ne, nd, frames, "gated edge fp16", block="gated")


@pytest.mark.parametrize("H,W,C,ne,nd", EDGE)
def test_gated_edge_shapes_int(H, W, C, ne, nd):
    frames = [synth.random_frame(H, W, seed=s) for s in (22, 23)]
    run_int_sequence(H, W, C, ne, nd, frames, "gated edge int", block="gated")


def test_gated_c256_ragged_fp16():
    """C = 256 gated blocks (the 128-pixels-per-wave kernel) over several ragged
    8 x 16 tiles (34 x 50 pixels at 1/8 scale) and 3 + 3 blocks, two frames."""
    frames = [synth.random_frame(272, 400, seed=s) for s in (24, 25)]
    run_fp16_sequence(272, 400, 256, 3, 3, frames, "gated c256 fp16", block="gated")


def test_gated_wvga_fp16():
    run_fp16_sequence(480, 832, 128, 6, 6, list(synth.frame_sequence("wvga", 1)), "gated wvga fp16", block="gated")


def test_gated_wvga_int_bit_exact():
    run_int_sequence(480, 832, 128, 6, 6, list(synth.frame_sequence("wvga", 2)), "gated wvga int", block="gated")


@pytest.mark.timeout(900)
def test_gated_hd1080_int_sampled_bit_exact():
    pre = synth.PRESETS["hd1080_int"]
    H, W, C, NE, ND, H16, W16, CROPS = geometry(pre)
    flat, p = params_for(C, NE, ND, "gated")
    ip = ci.integerize(p)
    enc = Codec(H, W, C, NE, ND, "int16", flat, device=DEV, block="gated")
    dec = Codec(H, W, C, NE, ND, "int16", flat, device=DEV, block="gated")
    x = next(iter(synth.frame_sequence(pre, 1)))
    say("gated 1080p int frame 0")
    f0, y0 = (host(v).astype(np.int64) for v in enc.get_state())
    q, _ = enc.encode(torch.from_numpy(x).to(DEV))
    xhat = host(dec.decode(q))
    f1, y1 = (host(v).astype(np.int64) for v in enc.get_state())
    d1, _ = (host(v).astype(np.int64) for v in dec.get_state())
    np.testing.assert_array_equal(d1, f1)
    qh = host(q).astype(np.int64)
    for (Y0, X0) in CROPS[1:]:
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
