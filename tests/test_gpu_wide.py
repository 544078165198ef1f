"""GPU parity of the wide DC blocks (C = 384, 512: the widths of a Large model,
supplementary "Performance for a Large Model", Tab. 8), which run as three
launches per block (depthwise; pw C -> 2C + LeakyReLU or the WSiLU gate of the
gated form; pw to C + residual).
Same bars as the other parity tests: int path free-running and bit-exact
(Alg. 1 for every convolution), fp16 teacher-forced within 2e-2 max(1, |ref|).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from oracle import codec_int as ci
from oracle import hyperprior as hp
from paper_2502_20762_amd.ncodec import Codec

from test_gpu_parity import gpu, host, run_fp16_sequence, run_int_sequence

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.mark.parametrize("C,H,W,ne,nd", [
    (384, 48, 80, 2, 1),     # 60 pixels at 1/8: one ragged tile
    (512, 112, 208, 1, 2),   # 364 pixels at 1/8: three tiles, ragged tail
])
def test_wide_blocks_fp16(C, H, W, ne, nd):
    frames = [synth.random_frame(H, W, seed=s) for s in (140, 141)]
    run_fp16_sequence(H, W, C, ne, nd, frames, f"wide fp16 C={C}")


@pytest.mark.parametrize("C,H,W,ne,nd", [
    (384, 48, 80, 2, 1),
    (512, 112, 208, 1, 2),
])
def test_wide_blocks_int_bit_exact(C, H, W, ne, nd):
    frames = [synth.random_frame(H, W, seed=s) for s in (142, 143)]
    run_int_sequence(H, W, C, ne, nd, frames, f"wide int C={C}")


@pytest.mark.parametrize("C", [384, 512])
def test_wide_gated_blocks_both_paths(C):
    # the gated form (Supp. B.1: WSiLU and Chunk; the int16 sigmoid table of Sec. 4.5)
    H, W, ne, nd = 48, 80, 1, 2
    frames = [synth.random_frame(H, W, seed=s) for s in (146, 147)]
    run_fp16_sequence(H, W, C, ne, nd, frames, f"wide gated fp16 C={C}", block="gated")
    run_int_sequence(H, W, C, ne, nd, frames, f"wide gated int C={C}", block="gated")


@pytest.mark.parametrize("path", ["fp16", "int16"])
def test_wide_kernels_per_frame(path):
    H, W, C, ne, nd = 32, 64, 512, 2, 1
    flat = synth.make_weights(C, ne, nd)
    enc = Codec(H, W, C, ne, nd, path, flat, device=DEV)
    dec = Codec(H, W, C, ne, nd, path, flat, device=DEV)
    enc.timing(True)
    dec.timing(True)
    q, _ = enc.encode(gpu(synth.random_frame(H, W, seed=144)))
    dec.decode(q)
    te, td = enc.timing_read(), dec.timing_read()
    enc.timing(False)
    dec.timing(False)
    fold = 1 if path == "fp16" else 0  # fp16: upsample + fuse and patch embed + fuse are one launch each
    assert enc.kernels_per_frame(False) == sum(n for n, _ in te.values()) == 6 - 2 * fold + 3 * (ne + nd)
    assert dec.kernels_per_frame(True) == sum(n for n, _ in td.values()) == 4 - fold + 3 * nd
    for kind in ("dcblock_dw", "dcblock_pw1", "dcblock_pw2"):
        assert te[kind][0] == ne + nd and td[kind][0] == nd


def test_wide_two_step_model_int_bit_exact():
    # the two-step entropy model at C = 512 (the second step's head is 256 -> 512)
    H, W, C, ne, nd = 64, 96, 512, 1, 1
    flat = synth.make_weights(C, ne, nd, hyper=True)
    p = oracle.unpack(flat, C, ne, nd, hyper=True)
    ip, ih = ci.integerize(p), hp.integerize_hyper(p)
    enc = Codec(H, W, C, ne, nd, "int16", flat, device=DEV, hyperprior=True)
    dec = Codec(H, W, C, ne, nd, "int16", flat, device=DEV, hyperprior=True)
    st = ci.zero_state(ip, H, W)
    ny = C * (H // 16) * (W // 16)
    for t in range(2):
        x = synth.random_frame(H, W, seed=145 + t)
        r = hp.encode_frame_int(p, ip, ih, x, st)
        q, bits = enc.encode(gpu(x))
        qh = host(q)
        np.testing.assert_array_equal(qh[:ny].reshape(r.sym.y().shape), r.sym.y())
        np.testing.assert_array_equal(qh[ny:].reshape(r.sym.qz.shape), r.sym.qz)
        assert abs(float(host(bits)) - r.bits) <= 1e-5 * r.bits
        xr, _ = hp.decode_frame_int(ip, ih, r.sym, st)
        np.testing.assert_array_equal(host(dec.decode(q)), xr)
        for a, b in zip(dec.get_state(), enc.get_state()):
            assert torch.equal(a, b)
        st = r.state
