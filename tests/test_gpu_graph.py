"""Graph replay against eager launches, through the C ABI.

A context with graph replay enabled replays a captured hipGraph per
(encode / decode, state buffer) and re-points the nodes that touch caller
buffers.  Each replay is checked against a second context that launches every
kernel directly (the default), with the program's own
eager work (state copies, torch ops, synchronisations) between the replays,
caller buffers that change from call to call, and calls without a bits
output.  Both paths run the same kernels, so the results must agree bitwise.
"""
import numpy as np
import pytest
import torch

import synth
from paper_2502_20762_amd.ncodec import Codec

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def say(*a):
    print("[gpu-graph]", *a, flush=True)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


GATED = dict(block="gated")
MODULES = dict(n_fe_blocks=1, n_rg_blocks=1, qp_banks=True)
HYPER = dict(hyperprior=True)  # the two-step entropy model: z symbols follow y's in q


@pytest.mark.parametrize("path,H,W,C,ne,nd,extra", [
    ("int16", 64, 64, 64, 2, 2, {}), ("fp16", 112, 208, 128, 2, 1, {}), ("int16", 48, 80, 128, 1, 2, {}),
    ("int16", 64, 96, 64, 1, 1, GATED), ("fp16", 64, 96, 64, 1, 1, MODULES),
    ("int16", 48, 80, 128, 1, 1, dict(GATED, **MODULES)), ("int16", 64, 96, 128, 1, 1, HYPER),
    ("fp16", 64, 96, 128, 1, 1, dict(HYPER, **MODULES)),
    # C = 256: block chains, the downsample inside the encoder's
    ("fp16", 112, 208, 256, 2, 2, {})])
def test_graph_replay_matches_eager(path, H, W, C, ne, nd, extra):
    block = extra.get("block", "lrelu")
    flat = synth.make_weights(C, ne, nd, block=block, n_fe=extra.get("n_fe_blocks", 0),
                              n_rg=extra.get("n_rg_blocks", 0), banks=extra.get("qp_banks", False),
                              hyper=extra.get("hyperprior", False))
    enc_g = Codec(H, W, C, ne, nd, path, flat, device=DEV, **extra)
    enc_e = Codec(H, W, C, ne, nd, path, flat, device=DEV, **extra)
    dec_g = Codec(H, W, C, ne, nd, path, flat, device=DEV, **extra)
    dec_e = Codec(H, W, C, ne, nd, path, flat, device=DEV, **extra)
    enc_g.graphs(True)
    dec_g.graphs(True)
    banks = extra.get("qp_banks", False)
    frames = [torch.from_numpy(synth.random_frame(H, W, seed=40 + s)).to(DEV) for s in range(6)]
    # two alternating sets of caller buffers, so the graph nodes are re-pointed
    qbuf = [torch.empty(enc_g.q_shape, dtype=torch.int16, device=DEV) for _ in range(2)]
    bbuf = [torch.zeros((), dtype=torch.float64, device=DEV) for _ in range(2)]
    odt = torch.int16 if path == "int16" else torch.float16
    obuf = [torch.empty(enc_g.frame_shape, dtype=odt, device=DEV) for _ in range(3)]
    for t, x in enumerate(frames):
        say(path, (H, W, C, ne, nd), extra, "frame", t)
        if banks and t == 3:  # a new rate point between replays: the weights change under the graphs
            for c in (enc_g, enc_e, dec_g, dec_e):
                c.set_qp(45)
        want_bits = t % 3 != 2
        qg, bg = enc_g.encode(x, q_out=qbuf[t % 2], bits_out=bbuf[t % 2] if want_bits else None,
                              want_bits=want_bits)
        qe, be = enc_e.encode(x, want_bits=want_bits)
        # eager work between replays
        fg, yg = enc_g.get_state()
        fe, ye = enc_e.get_state()
        _ = (x.float() * 0.5).sum()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(qg), host(qe), err_msg=f"{path} t={t} q")
        np.testing.assert_array_equal(host(fg), host(fe), err_msg=f"{path} t={t} f_t")
        np.testing.assert_array_equal(host(yg), host(ye), err_msg=f"{path} t={t} yhat")
        if want_bits:
            assert float(host(bg)) == float(host(be)), (t, float(host(bg)), float(host(be)))
        xg = dec_g.decode(qe, out=obuf[t % 3])
        xe = dec_e.decode(qe)
        np.testing.assert_array_equal(host(xg), host(xe), err_msg=f"{path} t={t} decoded frame")
        dfg, dyg = dec_g.get_state()
        np.testing.assert_array_equal(host(dfg), host(fe), err_msg=f"{path} t={t} decoder f_t")
    # reset between replays: the next frame is an I-frame on both
    enc_g.reset()
    enc_e.reset()
    qg, _ = enc_g.encode(frames[0], q_out=qbuf[1])
    qe, _ = enc_e.encode(frames[0])
    np.testing.assert_array_equal(host(qg), host(qe), err_msg=f"{path} after reset q")
