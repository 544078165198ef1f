"""Integerised transform of one frame, exact integer arithmetic.

Model integerisation (Sec. 4.5, Eq. 3; Supp. B.4, Alg. 1):

* features are int16 with v_i = round(K1 * v_f), K1 = 512 (Eq. 3); the input
  frame is converted once, x_i = round(512 x);
* every convolution uses int16 weights w_i = round(K2 w_f) and biases
  b_i = round(K2 b_f), K2 = 8192, accumulates a = conv(x_i, w_i) + b_i * K1 in
  int32 and returns clip(a / K2, -32768, 32767) (Alg. 1).

Readings (the paper gives no rounding mode for a / K2, no integer LeakyReLU,
residual or quantiser): every "round" and every division by a power of two is
round-half-to-even computed from floor and remainder; the LeakyReLU slope is
the K2 constant 819 = round(0.1 * 8192) followed by the same rescale; the
residual add saturates to int16; the quantiser is q = round((y_i - mu_i) / K1)
and yhat_i = clip(K1 q + mu_i).  An accumulator outside the int32 range raises
``OverflowError`` (the paper observes none, Sec. 4.5).

Pointwise and 2x2 contractions are evaluated with float64 matrix products on
integer-valued operands; :func:`int_matmul` checks first that every partial
sum is below 2^53, which makes the product exact in any summation order.
"""
from __future__ import annotations

import dataclasses

import numpy as np
from scipy.special import expit

from . import bits as _bits
from .ops import pixel_shuffle, pixel_unshuffle
from .params import Params

K1 = 512
K2_SHIFT = 13           # K2 = 8192
LRELU_SLOPE_I = 819     # round(0.1 * 8192)
INT16_MIN, INT16_MAX = -32768, 32767
INT32_LIMIT = 1 << 31


def rhe_shift(a: np.ndarray, s: int) -> np.ndarray:
    """round-half-to-even of a / 2^s for integer a (exact, from floor and remainder)."""
    a = np.asarray(a, dtype=np.int64)
    d = np.int64(1) << np.int64(s)
    fl = np.floor_divide(a, d)
    r = a - fl * d
    half = d // 2
    up = (r > half) | ((r == half) & (np.mod(fl, 2) == 1))
    return fl + up.astype(np.int64)


def clip16(v: np.ndarray) -> np.ndarray:
    return np.clip(v, INT16_MIN, INT16_MAX).astype(np.int64)


def quantize_param(v: np.ndarray) -> np.ndarray:
    """w_i = round(K2 w_f) as int16 (Alg. 1); K2 w_f is exact in float64."""
    return clip16(np.rint(np.asarray(v, dtype=np.float64) * (1 << K2_SHIFT)))


def frame_to_int(x: np.ndarray) -> np.ndarray:
    """x_i = round(K1 x) for the fp16 input frame (Alg. 1, first branch)."""
    return clip16(np.rint(np.asarray(x, dtype=np.float64) * K1))


def _check32(a: np.ndarray, what: str) -> None:
    if a.size and int(np.max(np.abs(a))) >= INT32_LIMIT:
        raise OverflowError(f"int32 accumulator overflow in {what}")


def int_matmul(w: np.ndarray, x: np.ndarray) -> np.ndarray:
    """Exact integer product w @ x (int64 result) via float64 BLAS."""
    K = w.shape[1]
    bound = K * max(int(np.max(np.abs(w), initial=0)), 1) * max(int(np.max(np.abs(x), initial=0)), 1)
    if bound >= (1 << 53):
        out = w.astype(object) @ x.astype(object)
        return np.asarray(out, dtype=np.int64)
    return (w.astype(np.float64) @ x.astype(np.float64)).astype(np.int64)


@dataclasses.dataclass
class IConv:
    w: np.ndarray  # int64 values in int16 range
    b: np.ndarray


def iconv(c) -> IConv:
    return IConv(quantize_param(c.w), quantize_param(c.b))


def rescale(a: np.ndarray, what: str) -> np.ndarray:
    _check32(a, what)
    return clip16(rhe_shift(a, K2_SHIFT))


def int_conv1x1(x: np.ndarray, c: IConv, what: str = "conv1x1") -> np.ndarray:
    K, h, w = x.shape
    a = int_matmul(c.w, x.reshape(K, h * w)) + K1 * c.b[:, None]
    return rescale(a, what).reshape(c.w.shape[0], h, w)


def int_dwconv3x3(x: np.ndarray, c: IConv) -> np.ndarray:
    C, H, W = x.shape
    pad = np.zeros((C, H + 2, W + 2), dtype=np.int64)
    pad[:, 1:H + 1, 1:W + 1] = x
    a = np.zeros((C, H, W), dtype=np.int64)
    for ky in range(3):
        for kx in range(3):
            a += c.w[:, ky, kx][:, None, None] * pad[:, ky:ky + H, kx:kx + W]
    a += K1 * c.b[:, None, None]
    return rescale(a, "dwconv3x3")


def int_conv2x2s2(x: np.ndarray, c: IConv) -> np.ndarray:
    C, H, W = x.shape
    a = np.zeros((c.w.shape[0], (H // 2) * (W // 2)), dtype=np.int64)
    for i in range(2):
        for j in range(2):
            a += int_matmul(c.w[:, :, i, j], x[:, i::2, j::2].reshape(C, -1))
    a += K1 * c.b[:, None]
    return rescale(a, "conv2x2s2").reshape(c.w.shape[0], H // 2, W // 2)


def int_leaky_relu(h: np.ndarray) -> np.ndarray:
    return np.where(h >= 0, h, rhe_shift(LRELU_SLOPE_I * h, K2_SHIFT))


_SIGMOID = None


def sigmoid_table() -> np.ndarray:
    """The int16 -> int16 sigmoid table of the integer WSiLU (Sec. 4.5: a
    precomputed lookup table handles the sigmoid): entry v + 32768 is
    round(K1 * sigmoid(4 v / K1)), the sigmoid of the K1-scaled input with the
    WSiLU weight alpha = 4 (Supp. B.1), itself K1-scaled (0 .. 512)."""
    global _SIGMOID
    if _SIGMOID is None:
        v = np.arange(-32768, 32768, dtype=np.float64)
        _SIGMOID = np.rint(K1 * expit(4.0 * v / K1)).astype(np.int64)
    return _SIGMOID


def int_wsilu(h: np.ndarray) -> np.ndarray:
    """round(h * S[h] / K1): |h S[h]| <= 2^24, the result is within int16."""
    return rhe_shift(h * sigmoid_table()[h + 32768], 9)


def int_gate(h1: np.ndarray, h2: np.ndarray) -> np.ndarray:
    """clip(round(WSiLU(h1) * h2 / K1)): the product of two K1-scaled values
    rescaled by K1 (|product| < 2^30)."""
    return clip16(rhe_shift(int_wsilu(h1) * h2, 9))


@dataclasses.dataclass
class IBlock:
    dw: IConv
    pw1: IConv
    pw2: IConv
    kind: str = "lrelu"


@dataclasses.dataclass
class IParams:
    C: int
    pe: IConv
    fuse_enc: IConv
    enc: list
    down: IConv
    head: IConv
    up: IConv
    fuse_dec: IConv
    dec: list
    rec: IConv
    fe: list = dataclasses.field(default_factory=list)
    rg: list = dataclasses.field(default_factory=list)


def integerize(p: Params) -> IParams:
    """Integer weights of p (fold the vector banks first: integerize(fold_qp(p, qp)))."""
    blk = lambda b: IBlock(iconv(b.dw), iconv(b.pw1), iconv(b.pw2), b.kind)  # noqa: E731
    return IParams(p.C, iconv(p.pe), iconv(p.fuse_enc), [blk(b) for b in p.enc],
                   iconv(p.down), iconv(p.head), iconv(p.up), iconv(p.fuse_dec),
                   [blk(b) for b in p.dec], iconv(p.rec), [blk(b) for b in p.fe], [blk(b) for b in p.rg])


@dataclasses.dataclass
class State:
    feat: np.ndarray
    yhat: np.ndarray


def zero_state(ip: IParams, height: int, width: int) -> State:
    C = ip.C
    return State(np.zeros((C, height // 8, width // 8), dtype=np.int64),
                 np.zeros((C, height // 16, width // 16), dtype=np.int64))


def dc_block(z: np.ndarray, b: IBlock) -> np.ndarray:
    a = int_dwconv3x3(z, b.dw)
    h = int_conv1x1(a, b.pw1, "pw1")
    if b.kind == "gated":
        C = z.shape[0]
        g = int_gate(h[:C], h[C:])
    else:
        g = int_leaky_relu(h)
    p = int_conv1x1(g, b.pw2, "pw2")
    return clip16(z + p)


def context(ip: IParams, f_prev: np.ndarray) -> np.ndarray:
    z = f_prev
    for b in ip.fe:
        z = dc_block(z, b)
    return z


def encoder_feature(ip: IParams, x: np.ndarray, f_prev: np.ndarray) -> np.ndarray:
    u = pixel_unshuffle(frame_to_int(x), 8)
    e = int_conv1x1(u, ip.pe, "patch embed")
    z = int_conv1x1(np.concatenate([e, context(ip, f_prev)], axis=0), ip.fuse_enc, "fuse_enc")
    for b in ip.enc:
        z = dc_block(z, b)
    return z


def analysis(ip: IParams, x: np.ndarray, f_prev: np.ndarray) -> np.ndarray:
    return int_conv2x2s2(encoder_feature(ip, x, f_prev), ip.down)


def prior(ip: IParams, yhat_prev: np.ndarray):
    ms = int_conv1x1(yhat_prev, ip.head, "head")
    return ms[:ip.C], ms[ip.C:]


def quantize(y: np.ndarray, mu: np.ndarray):
    q = rhe_shift(y - mu, 9)          # divide by K1 = 2^9
    return q, clip16(K1 * q + mu)


def sigma_int(s: np.ndarray) -> np.ndarray:
    return _bits.sigma_from_s(np.asarray(s, dtype=np.float64) / K1)


def decoder_feature(ip: IParams, yhat: np.ndarray, f_prev: np.ndarray) -> np.ndarray:
    d = pixel_shuffle(int_conv1x1(yhat, ip.up, "up"), 2)
    z = int_conv1x1(np.concatenate([d, context(ip, f_prev)], axis=0), ip.fuse_dec, "fuse_dec")
    for b in ip.dec:
        z = dc_block(z, b)
    return z


def reconstruct(ip: IParams, f: np.ndarray) -> np.ndarray:
    for b in ip.rg:
        f = dc_block(f, b)
    r = int_conv1x1(f, ip.rec, "rec")
    return np.clip(pixel_shuffle(r, 8), 0, K1).astype(np.int64)


@dataclasses.dataclass
class EncodeResult:
    q: np.ndarray
    bits: float
    y: np.ndarray
    mu: np.ndarray
    s: np.ndarray
    state: State


def encode_frame(ip: IParams, x: np.ndarray, state: State) -> EncodeResult:
    y = analysis(ip, x, state.feat)
    mu, s = prior(ip, state.yhat)
    q, yhat = quantize(y, mu)
    nbits = _bits.estimate_bits(q, sigma_int(s))
    f_t = decoder_feature(ip, yhat, state.feat)
    return EncodeResult(q, nbits, y, mu, s, State(f_t, yhat))


def decode_frame(ip: IParams, q: np.ndarray, state: State):
    mu, _ = prior(ip, state.yhat)
    yhat = clip16(K1 * np.asarray(q, dtype=np.int64) + mu)
    f_t = decoder_feature(ip, yhat, state.feat)
    return reconstruct(ip, f_t), State(f_t, yhat)
