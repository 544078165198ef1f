"""Two-step entropy model with a hyperprior z (TEST INFRASTRUCTURE, like the
rest of ``oracle``): float64 and exact-integer forms.

The paper codes a hyper latent z besides y (Sec. 4.4: z carries more than 10 %
of y's bits, so its distribution comes from a bank of factorized modules, one
per rate point) and estimates y's distribution in two steps (supplementary,
"Entropy model"): the decoder decodes z, estimates the distribution, decodes
the first part y^1, then the second part y^2 (supplementary, "Parallel
Coding").  The paper gives the roles, not the layers; the readings here (H1-H7
in the design doc) are:

* hyper-analysis   z = conv2x2/s2(y) (C -> CZ = 64 channels, 1/32 scale);
* quantisation     q_z = round(z), zhat = q_z (int: q_z = round(z_i / 512),
                   zhat_i = clip(512 q_z)), coded under a zero-mean Gaussian
                   per channel whose scale comes from the z bank row of the
                   rate point (the nearest row for a rate between two points);
* hyper-synthesis  [mu_h ; s_h] = shuffle2(W_zs zhat + b) (2C channels, 1/16);
* step 1           [mu ; s] = prior(yhat_{t-1}) + [mu_h ; s_h] (int: a
                   saturating add); the first C/2 channels y^1 are quantised
                   with (mu, s) of those channels;
* step 2           [dmu ; ds] = W_2 yhat^1 + b (C/2 -> C); the last C/2
                   channels y^2 use mu^2 = mu + dmu, s^2 = s + ds;
* rate             bits(z) + bits(y^1) + bits(y^2), each -log2 of the
                   Gaussian likelihood of Supp. B.2 (``bits``).

Everything else of the transform is ``codec_float`` / ``codec_int``.
Parity status: pinned by tests/test_oracle_hyperprior.py (reduction to the
one-step model, brute-force Fraction evaluation of the integer steps,
encoder/decoder agreement, rate decomposition).
"""
from __future__ import annotations

import dataclasses

import numpy as np

from . import bits as _bits
from . import codec_float as cf
from . import codec_int as ci
from .ops import conv1x1, conv2x2s2, pixel_shuffle
from .params import NUM_QP, Params


def z_row(qp) -> int:
    """Row of the z bank for rate point qp in [0, 63]: the nearest learned
    point (supplementary, rate adjustment: the factorized module is the
    nearest one, not an interpolation); a tie rounds up."""
    qp = float(qp)
    if not 0.0 <= qp <= NUM_QP - 1:
        raise ValueError(f"qp must be in [0, {NUM_QP - 1}]")
    return int(np.floor(qp + 0.5))


def z_sigma(p: Params, qp=0) -> np.ndarray:
    """Scale of every z channel at rate point qp (the bank row, floored at
    the minimum scale of the rate model)."""
    return np.maximum(np.asarray(p.hyper.zbank[z_row(qp)], np.float64), _bits.SIGMA_MIN)


@dataclasses.dataclass
class Symbols:
    qz: np.ndarray   # CZ x H/32 x W/32
    q1: np.ndarray   # C/2 x H/16 x W/16
    q2: np.ndarray   # C/2 x H/16 x W/16

    def y(self) -> np.ndarray:
        return np.concatenate([self.q1, self.q2], axis=0)


@dataclasses.dataclass
class Encoded:
    sym: Symbols
    bits: float
    bits_z: float
    bits_y1: float
    bits_y2: float
    sigma1: np.ndarray
    sigma2: np.ndarray
    state: object


# ------------------------------------------------------------------ float path
def hyper_params_float(p: Params, zhat: np.ndarray):
    hp = pixel_shuffle(conv1x1(zhat, p.hyper.zsyn.w, p.hyper.zsyn.b), 2)
    return hp[:p.C], hp[p.C:]


def step2_float(p: Params, yhat1: np.ndarray):
    d = conv1x1(yhat1, p.hyper.step2.w, p.hyper.step2.b)
    return d[:p.C // 2], d[p.C // 2:]


def two_step_float(p: Params, y: np.ndarray, yhat_prev: np.ndarray):
    """The entropy model on the latent y: (symbols, yhat, sigma^1, sigma^2)."""
    H2 = p.C // 2
    z = conv2x2s2(y, p.hyper.zana.w, p.hyper.zana.b)
    qz = np.rint(z)                       # round half to even
    mu_h, s_h = hyper_params_float(p, qz)
    mu_t, s_t = cf.prior(p, yhat_prev)
    mu, s = mu_t + mu_h, s_t + s_h
    q1 = np.rint(y[:H2] - mu[:H2])
    yhat1 = q1 + mu[:H2]
    dmu, ds = step2_float(p, yhat1)
    mu2, s2 = mu[H2:] + dmu, s[H2:] + ds
    q2 = np.rint(y[H2:] - mu2)
    yhat = np.concatenate([yhat1, q2 + mu2], axis=0)
    sym = Symbols(qz.astype(np.int64), q1.astype(np.int64), q2.astype(np.int64))
    return sym, yhat, _bits.sigma_from_s(s[:H2]), _bits.sigma_from_s(s2)


def rates(p: Params, sym: Symbols, sig1: np.ndarray, sig2: np.ndarray, qp=0):
    """(bits of z, of y^1, of y^2)."""
    qz = np.asarray(sym.qz, np.float64)
    bz = _bits.estimate_bits(qz, z_sigma(p, qp)[:, None, None] * np.ones(qz.shape))
    return bz, _bits.estimate_bits(sym.q1, sig1), _bits.estimate_bits(sym.q2, sig2)


def encode_frame_float(p: Params, x: np.ndarray, state: cf.State, qp=0) -> Encoded:
    y = cf.analysis(p, x, state.feat)
    sym, yhat, sig1, sig2 = two_step_float(p, y, state.yhat)
    bz, b1, b2 = rates(p, sym, sig1, sig2, qp)
    f_t = cf.decoder_feature(p, yhat, state.feat)
    return Encoded(sym, bz + b1 + b2, bz, b1, b2, sig1, sig2, cf.State(f_t, yhat))


def latent_from_symbols_float(p: Params, sym: Symbols, yhat_prev: np.ndarray):
    """yhat and the two steps' scales, from the symbols (the decoder's order:
    z, then the distribution, then y^1, then y^2)."""
    H2 = p.C // 2
    mu_h, s_h = hyper_params_float(p, np.asarray(sym.qz, np.float64))
    mu_t, s_t = cf.prior(p, yhat_prev)
    mu, s = mu_t + mu_h, s_t + s_h
    yhat1 = np.asarray(sym.q1, np.float64) + mu[:H2]
    dmu, ds = step2_float(p, yhat1)
    mu2 = mu[H2:] + dmu                   # the encoder's operation order
    yhat2 = np.asarray(sym.q2, np.float64) + mu2
    return np.concatenate([yhat1, yhat2], axis=0), _bits.sigma_from_s(s[:H2]), _bits.sigma_from_s(s[H2:] + ds)


def decode_frame_float(p: Params, sym: Symbols, state: cf.State):
    yhat, _, _ = latent_from_symbols_float(p, sym, state.yhat)
    f_t = cf.decoder_feature(p, yhat, state.feat)
    return cf.reconstruct(p, f_t), cf.State(f_t, yhat)


# ------------------------------------------------------------------ int path
@dataclasses.dataclass
class IHyper:
    zana: ci.IConv
    zsyn: ci.IConv
    step2: ci.IConv


def integerize_hyper(p: Params) -> IHyper:
    h = p.hyper
    return IHyper(ci.iconv(h.zana), ci.iconv(h.zsyn), ci.iconv(h.step2))


def hyper_params_int(ih: IHyper, C: int, zhat: np.ndarray):
    hp = pixel_shuffle(ci.int_conv1x1(zhat, ih.zsyn, "hyper-synthesis"), 2)
    return hp[:C], hp[C:]


def step2_int(ih: IHyper, C: int, yhat1: np.ndarray):
    d = ci.int_conv1x1(yhat1, ih.step2, "step 2")
    return d[:C // 2], d[C // 2:]


def two_step_int(ip: ci.IParams, ih: IHyper, y: np.ndarray, yhat_prev: np.ndarray):
    """The entropy model on the integer latent y: (symbols, yhat, sigma^1, sigma^2)."""
    C = ip.C
    H2 = C // 2
    z = ci.int_conv2x2s2(y, ih.zana)
    qz = ci.rhe_shift(z, 9)                 # round(z_i / K1)
    zhat = ci.clip16(ci.K1 * qz)
    mu_h, s_h = hyper_params_int(ih, C, zhat)
    mu_t, s_t = ci.prior(ip, yhat_prev)
    mu, s = ci.clip16(mu_t + mu_h), ci.clip16(s_t + s_h)
    q1, yhat1 = ci.quantize(y[:H2], mu[:H2])
    dmu, ds = step2_int(ih, C, yhat1)
    mu2, s2 = ci.clip16(mu[H2:] + dmu), ci.clip16(s[H2:] + ds)
    q2, yhat2 = ci.quantize(y[H2:], mu2)
    return Symbols(qz, q1, q2), np.concatenate([yhat1, yhat2], axis=0), ci.sigma_int(s[:H2]), ci.sigma_int(s2)


def encode_frame_int(p: Params, ip: ci.IParams, ih: IHyper, x: np.ndarray, state: ci.State, qp=0) -> Encoded:
    y = ci.analysis(ip, x, state.feat)
    sym, yhat, sig1, sig2 = two_step_int(ip, ih, y, state.yhat)
    bz, b1, b2 = rates(p, sym, sig1, sig2, qp)
    f_t = ci.decoder_feature(ip, yhat, state.feat)
    return Encoded(sym, bz + b1 + b2, bz, b1, b2, sig1, sig2, ci.State(f_t, yhat))


def latent_from_symbols_int(ip: ci.IParams, ih: IHyper, sym: Symbols, yhat_prev: np.ndarray):
    C = ip.C
    H2 = C // 2
    zhat = ci.clip16(ci.K1 * np.asarray(sym.qz, np.int64))
    mu_h, s_h = hyper_params_int(ih, C, zhat)
    mu_t, s_t = ci.prior(ip, yhat_prev)
    mu, s = ci.clip16(mu_t + mu_h), ci.clip16(s_t + s_h)
    yhat1 = ci.clip16(ci.K1 * np.asarray(sym.q1, np.int64) + mu[:H2])
    dmu, ds = step2_int(ih, C, yhat1)
    mu2, s2 = ci.clip16(mu[H2:] + dmu), ci.clip16(s[H2:] + ds)
    yhat2 = ci.clip16(ci.K1 * np.asarray(sym.q2, np.int64) + mu2)
    return np.concatenate([yhat1, yhat2], axis=0), ci.sigma_int(s[:H2]), ci.sigma_int(s2)


def decode_frame_int(ip: ci.IParams, ih: IHyper, sym: Symbols, state: ci.State):
    yhat, _, _ = latent_from_symbols_int(ip, ih, sym, state.yhat)
    f_t = ci.decoder_feature(ip, yhat, state.feat)
    return ci.reconstruct(ip, f_t), ci.State(f_t, yhat)
