"""Floating-point transform of one frame, float64 throughout.

Follows the paper's framework (Sec. 4.1 and Fig. 4): the frame is
patch-embedded straight to 1/8 resolution (Sec. 4.2), the previous decoded
feature is concatenated on channels as the temporal context (Sec. 4.3), the
encoder and decoder are stacks of depth-wise conv blocks at that single scale
(Supp. B.1), and the latent is quantised and its rate estimated (Fig. 4 "Q",
Supp. B.2).  The reference feature for the next frame is the decoder output
before reconstruction (Supp. B.3), so encoding runs the decoder too but not
the reconstruction head.

Readings where the paper is silent (block internals, fuse conv, 1/16 latent,
prior input, sigma mapping) are listed in the design doc.

State is (f_prev: C x H/8 x W/8, yhat_prev: C x H/16 x W/16); zeros for an
I-frame.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from . import bits as _bits
from .ops import (conv1x1, conv2x2s2, dwconv3x3, leaky_relu, pixel_shuffle,
                  pixel_unshuffle, wsilu)
from .params import Params


@dataclasses.dataclass
class State:
    feat: np.ndarray   # f_{t-1}
    yhat: np.ndarray   # yhat_{t-1}


def zero_state(p: Params, height: int, width: int) -> State:
    C = p.C
    return State(np.zeros((C, height // 8, width // 8)),
                 np.zeros((C, height // 16, width // 16)))


def dc_block(z: np.ndarray, blk) -> np.ndarray:
    """LeakyReLU block: z + pw2(LeakyReLU_0.1(pw1(dw3x3(z)))).
    Gated block (Supp. B.1: WSiLU, Chunk): h = pw1(dw3x3(z)) is chunked on
    channels into (h1, h2) and z + pw2(WSiLU(h1) * h2)."""
    a = dwconv3x3(z, blk.dw.w, blk.dw.b)
    h = conv1x1(a, blk.pw1.w, blk.pw1.b)
    if blk.kind == "gated":
        C = z.shape[0]
        g = wsilu(h[:C]) * h[C:]
    else:
        g = leaky_relu(h, 0.1)
    return z + conv1x1(g, blk.pw2.w, blk.pw2.b)


def context(p: Params, f_prev: np.ndarray) -> np.ndarray:
    """Temporal context F_{t-1}: the feature extractor's blocks on f_{t-1}
    (f_{t-1} itself without a feature extractor)."""
    z = f_prev
    for blk in p.fe:
        z = dc_block(z, blk)
    return z


def encoder_feature(p: Params, x: np.ndarray, f_prev: np.ndarray) -> np.ndarray:
    """Patch embed, concatenate context, fuse, N_e blocks (the analysis transform at 1/8)."""
    u = pixel_unshuffle(np.asarray(x, dtype=np.float64), 8)
    e = conv1x1(u, p.pe.w, p.pe.b)
    z = conv1x1(np.concatenate([e, context(p, f_prev)], axis=0), p.fuse_enc.w, p.fuse_enc.b)
    for blk in p.enc:
        z = dc_block(z, blk)
    return z


def analysis(p: Params, x: np.ndarray, f_prev: np.ndarray) -> np.ndarray:
    """Latent y at 1/16 resolution."""
    z = encoder_feature(p, x, f_prev)
    return conv2x2s2(z, p.down.w, p.down.b)


def prior(p: Params, yhat_prev: np.ndarray):
    """mu, s from a 1x1 head on the previous frame's quantised latent."""
    ms = conv1x1(yhat_prev, p.head.w, p.head.b)
    return ms[:p.C], ms[p.C:]


def decoder_feature(p: Params, yhat: np.ndarray, f_prev: np.ndarray) -> np.ndarray:
    """Upsample to 1/8, concatenate context, fuse, N_d blocks -> f_t."""
    d = pixel_shuffle(conv1x1(yhat, p.up.w, p.up.b), 2)
    z = conv1x1(np.concatenate([d, context(p, f_prev)], axis=0), p.fuse_dec.w, p.fuse_dec.b)
    for blk in p.dec:
        z = dc_block(z, blk)
    return z


def reconstruct(p: Params, f: np.ndarray) -> np.ndarray:
    """Reconstruction generation blocks on f_t, then the reconstruction conv."""
    for blk in p.rg:
        f = dc_block(f, blk)
    r = conv1x1(f, p.rec.w, p.rec.b)
    return np.clip(pixel_shuffle(r, 8), 0.0, 1.0)


@dataclasses.dataclass
class EncodeResult:
    q: np.ndarray
    bits: float
    y: np.ndarray
    mu: np.ndarray
    sigma: np.ndarray
    state: State


def encode_frame(p: Params, x: np.ndarray, state: State) -> EncodeResult:
    y = analysis(p, x, state.feat)
    mu, s = prior(p, state.yhat)
    q = np.rint(y - mu)                      # round half to even
    yhat = q + mu
    sigma = _bits.sigma_from_s(s)
    nbits = _bits.estimate_bits(q, sigma)
    f_t = decoder_feature(p, yhat, state.feat)
    return EncodeResult(q.astype(np.int64), nbits, y, mu, sigma, State(f_t, yhat))


def decode_frame(p: Params, q: np.ndarray, state: State):
    """Returns (xhat in [0,1], new state)."""
    mu, _ = prior(p, state.yhat)
    yhat = np.asarray(q, dtype=np.float64) + mu
    f_t = decoder_feature(p, yhat, state.feat)
    return reconstruct(p, f_t), State(f_t, yhat)
