"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This module draws random numbers and nothing else: it holds none of the
codec's arithmetic (no convolution, quantisation or likelihood).  Both the CPU
oracle and the GPU library consume exactly the arrays produced here.

Inputs are stand-ins for the paper's speed workloads (1920x1080, 3840x2160
and smaller sequences from public test sets, Sec. 5.1 "Test Details"): RGB in
[0, 1], smooth content with small global motion, as in low-delay P-frame
coding.  No dataset item is reproduced.

Weights are random-init (no trained model exists here).  The canonical flat
parameter order is the interface of ``ncodec_create`` and is documented in
``include/ncodec.h``; the list below only fixes the order in which values are
drawn.
"""
from __future__ import annotations

import dataclasses

import numpy as np

SEED_W = 0  # weights
SEED_X = 1  # frames

# Gain applied to the second pointwise conv of every residual block (the
# projection that feeds the residual add).  With plain N(0, 1/fan_in) on that
# projection each block multiplies the residual stream's energy by about 1.5,
# and because the decoded feature is fed back as the next frame's context the
# recursion over frames diverges (past the int16 range at K1 = 512 within a few
# frames).  A trained codec keeps features inside [-64, 64) (Sec. 4.5); this
# down-scaled projection keeps the random-init transform inside that range
# over 32 frames.
RESID_GAIN = 0.125


@dataclasses.dataclass(frozen=True)
class Preset:
    name: str
    height: int
    width: int
    channels: int
    n_enc: int
    n_dec: int
    path: str  # "fp16" or "int16"
    n_frames: int
    frames: str  # "uniform" | "smooth" | "shifted"


PRESETS = {
    # 3x64x64 I/P pair, U[0,1] pixels.
    "tiny": Preset("tiny", 64, 64, 64, 2, 2, "fp16", 2, "uniform"),
    "tiny_int": Preset("tiny_int", 64, 64, 64, 2, 2, "int16", 2, "uniform"),
    # one 832x480 smooth frame, C=128, 6+6 blocks.
    "wvga": Preset("wvga", 480, 832, 128, 6, 6, "fp16", 1, "smooth"),
    # 1920x1088 (1080p padded to x16), C=256, 8+8 blocks, 32 shifted frames.
    "hd1080": Preset("hd1080", 1088, 1920, 256, 8, 8, "fp16", 32, "shifted"),
    "hd1080_int": Preset("hd1080_int", 1088, 1920, 256, 8, 8, "int16", 32, "shifted"),
    # 3840x2176 (2160p padded), 16 shifted frames.
    "uhd4k": Preset("uhd4k", 2176, 3840, 256, 8, 8, "fp16", 16, "shifted"),
}


CZ = 64  # channels of the hyper latent z (two-step entropy model)


def param_list(channels: int, n_enc: int, n_dec: int, block: str = "lrelu",
               n_fe: int = 0, n_rg: int = 0, banks: bool = False, hyper: bool = False):
    """(name, shape, fan_in, kind) in canonical order; kind is 'w', 'w_res', 'b'
    or 'bank'.

    ``block`` is the DC-block form: "lrelu" (pw2 is C x 2C) or "gated" (the
    hidden 2C channels are chunked into two halves and gated, pw2 is C x C).
    After the transform come ``n_fe`` feature-extractor blocks, ``n_rg``
    reconstruction-generation blocks and, with ``banks``, the four qp-indexed
    vector banks q_e, q_d, q_f, q_r (64 rate points x C each) and, with
    ``hyper``, the two-step entropy model: hyper-analysis zana (CZ x C x 2 x 2),
    hyper-synthesis zsyn (8C x CZ), second-step head step2 (C x C/2) and the
    bank of z scales zbank (64 rate points x CZ)."""
    C = channels
    out = []
    if block not in ("lrelu", "gated"):
        raise ValueError(f"unknown block form {block!r}")
    hid = 2 * C if block == "lrelu" else C

    def conv(name, wshape, fan_in, kind="w"):
        out.append((name + ".w", wshape, fan_in, kind))
        out.append((name + ".b", (wshape[0],), fan_in, "b"))

    def block_params(prefix):
        conv(prefix + ".dw", (C, 3, 3), 9)
        conv(prefix + ".pw1", (2 * C, C), C)
        conv(prefix + ".pw2", (C, hid), hid, "w_res")

    conv("pe", (C, 192), 192)
    conv("fuse_enc", (C, 2 * C), 2 * C)
    for k in range(n_enc):
        block_params(f"enc{k}")
    conv("down", (C, C, 2, 2), 4 * C)
    conv("head", (2 * C, C), C)
    conv("up", (4 * C, C), C)
    conv("fuse_dec", (C, 2 * C), 2 * C)
    for k in range(n_dec):
        block_params(f"dec{k}")
    conv("rec", (192, C), C)
    for k in range(n_fe):
        block_params(f"fe{k}")
    for k in range(n_rg):
        block_params(f"rg{k}")
    if banks:
        for name in ("q_e", "q_d", "q_f", "q_r"):
            out.append((name, (NUM_QP, C), 0, "bank"))
    if hyper:
        conv("zana", (CZ, C, 2, 2), 4 * C)
        conv("zsyn", (8 * C, CZ), CZ)
        conv("step2", (C, C // 2), C // 2)
        out.append(("zbank", (NUM_QP, CZ), 0, "zbank"))
    return out


NUM_QP = 64  # rate points of the vector banks


def bank_values(rng: np.random.Generator, name: str, channels: int) -> np.ndarray:
    """Synthetic vector banks: row qp scales the encoder output by about
    2^(-qp / 32) (coarser quantisation at higher qp) and the decoder input by the
    inverse; the context and reconstruction banks stay near 1; every entry
    carries a +-10 % per-channel jitter."""
    qp = np.arange(NUM_QP, dtype=np.float64)[:, None]
    jit = np.exp(rng.uniform(-0.1, 0.1, size=(NUM_QP, channels)))
    if name == "q_e":
        return 2.0 ** (-qp / 32.0) * jit
    if name == "zbank":  # scale of z: about 2 at qp 0, falling with the rate
        return 2.0 * 2.0 ** (-qp / 32.0) * jit
    if name == "q_d":
        return 2.0 ** (qp / 32.0) * jit
    return jit


def make_weights(channels: int, n_enc: int, n_dec: int, seed: int = SEED_W,
                 resid_gain: float = RESID_GAIN, block: str = "lrelu",
                 n_fe: int = 0, n_rg: int = 0, banks: bool = False, hyper: bool = False) -> np.ndarray:
    """Flat float32 parameter vector; every value is exactly fp16-representable.

    Weights ~ N(0, 1/fan_in) (the residual projection times ``resid_gain``),
    biases ~ U(-0.1, 0.1); each value is rounded to fp16 once.
    """
    rng = np.random.default_rng(seed)
    chunks = []
    for name, shape, fan_in, kind in param_list(channels, n_enc, n_dec, block, n_fe, n_rg, banks, hyper):
        if kind == "bank":
            chunks.append(bank_values(rng, name, channels).reshape(-1))
            continue
        if kind == "zbank":
            chunks.append(bank_values(rng, name, shape[1]).reshape(-1))
            continue
        if kind == "b":
            v = rng.uniform(-0.1, 0.1, size=shape)
        else:
            std = (1.0 / fan_in) ** 0.5
            if kind == "w_res":
                std *= resid_gain
            v = rng.standard_normal(size=shape) * std
        chunks.append(v.reshape(-1))
    flat = np.concatenate(chunks)
    return flat.astype(np.float16).astype(np.float32)


def smooth_frame(rng: np.random.Generator, height: int, width: int) -> np.ndarray:
    """3xHxW float64 in [0,1]: 0.5 + 8 random 2D sinusoids per channel + N(0, 0.02^2)."""
    yy = np.arange(height, dtype=np.float64)[:, None] / height
    xx = np.arange(width, dtype=np.float64)[None, :] / width
    out = np.empty((3, height, width), dtype=np.float64)
    for c in range(3):
        s = np.full((height, width), 0.5)
        a = rng.uniform(0.02, 0.08, size=8)
        fx = rng.uniform(-8.0, 8.0, size=8)
        fy = rng.uniform(-8.0, 8.0, size=8)
        ph = rng.uniform(0.0, 2.0 * np.pi, size=8)
        for k in range(8):
            s += a[k] * np.sin(2.0 * np.pi * (fx[k] * xx + fy[k] * yy) + ph[k])
        out[c] = s
    out += rng.normal(0.0, 0.02, size=out.shape)
    return np.clip(out, 0.0, 1.0)


def frame_sequence(preset: Preset | str, n_frames: int | None = None,
                   seed: int = SEED_X):
    """Yield fp16 frames (3,H,W) of the preset's workload, deterministically."""
    if isinstance(preset, str):
        preset = PRESETS[preset]
    n = preset.n_frames if n_frames is None else n_frames
    rng = np.random.default_rng(seed)
    H, W = preset.height, preset.width
    if preset.frames == "uniform":
        for _ in range(n):
            yield rng.uniform(0.0, 1.0, size=(3, H, W)).astype(np.float16)
        return
    x = smooth_frame(rng, H, W)
    for t in range(n):
        if t > 0:
            dx, dy = rng.integers(-4, 5, size=2)
            x = np.roll(x, shift=(int(dy), int(dx)), axis=(1, 2))
            x = np.clip(x + rng.normal(0.0, 0.01, size=x.shape), 0.0, 1.0)
        yield x.astype(np.float16)


def random_frame(height: int, width: int, seed: int) -> np.ndarray:
    """One U[0,1] fp16 frame for edge-case tests."""
    rng = np.random.default_rng(seed)
    return rng.uniform(0.0, 1.0, size=(3, height, width)).astype(np.float16)
