"""The oracle's own reading of the canonical flat parameter list.

Order (each weight row-major, each followed by its bias):
  pe        W(C,192)   b(C)
  fuse_enc  W(C,2C)    b(C)      input channels [e ; f_prev]
  enc[k]    dw W(C,3,3) b(C); pw1 W(2C,C) b(2C); pw2 W(C,H) b(C)    k < N_e
            (H = 2C for the LeakyReLU block, C for the gated block)
  down      W(C,C,2,2) b(C)
  head      W(2C,C)    b(2C)     rows [mu ; s]
  up        W(4C,C)    b(4C)     row 4c+2i+j -> pixel-shuffle position (c,i,j)
  fuse_dec  W(C,2C)    b(C)      input channels [d ; f_prev]
  dec[k]    as enc[k]                                                k < N_d
  rec       W(192,C)   b(192)    row 64c+8i+j -> colour c at (8y+i, 8x+j)
  fe[k]     as enc[k]                                                k < N_f
  rg[k]     as enc[k]                                                k < N_r
  q_e, q_d, q_f, q_r   (64, C) each, only with vector banks
  then, only with the two-step entropy model (``hyper``):
  zana      W(CZ,C,2,2) b(CZ)    hyper-analysis y -> z at 1/32
  zsyn      W(8C,CZ)    b(8C)    hyper-synthesis, row 4m+2i+j -> pixel-shuffle
                                 position (m,i,j) of the 2C hyper channels [mu ; s]
  step2     W(C,C/2)    b(C)     second step: rows [dmu ; ds] for the last C/2
                                 channels, from the first C/2 channels of yhat
  zbank     (64, CZ)             scale of z per channel at each rate point (> 0)

The conditional-coding modules (Fig. 4; Sec. 4.3, 4.4): the feature extractor
fe turns f_{t-1} into the temporal context F_{t-1} that both fuse convs take
in place of f_{t-1}; the reconstruction generation rg runs on f_t before the
reconstruction conv; the vector banks (Sec. 4.4) hold one per-channel scale
vector per rate point qp for the encoder output (q_e), the decoder input
(q_d), the extracted context (q_f) and the reconstruction input (q_r).
:func:`fold_qp` applies row qp of the banks to the adjacent convolutions.
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass
class Conv:
    w: np.ndarray
    b: np.ndarray


@dataclasses.dataclass
class Block:
    dw: Conv
    pw1: Conv
    pw2: Conv
    kind: str = "lrelu"   # "lrelu" or "gated"


CZ = 64  # channels of the hyper latent z


@dataclasses.dataclass
class Hyper:
    zana: Conv
    zsyn: Conv
    step2: Conv
    zbank: np.ndarray   # (64, CZ)


@dataclasses.dataclass
class Params:
    C: int
    pe: Conv
    fuse_enc: Conv
    enc: list
    down: Conv
    head: Conv
    up: Conv
    fuse_dec: Conv
    dec: list
    rec: Conv
    block: str = "lrelu"
    fe: list = dataclasses.field(default_factory=list)
    rg: list = dataclasses.field(default_factory=list)
    banks: dict = None    # name -> (64, C) array, or None
    hyper: Hyper = None   # the two-step entropy model with hyperprior, or None


NUM_QP = 64


def _hidden(C: int, block: str) -> int:
    if block not in ("lrelu", "gated"):
        raise ValueError(f"unknown block form {block!r}")
    return 2 * C if block == "lrelu" else C


def hyper_count(C: int) -> int:
    return CZ * C * 4 + CZ + 8 * C * CZ + 8 * C + C * (C // 2) + C + NUM_QP * CZ


def count(C: int, n_enc: int, n_dec: int, block: str = "lrelu", n_fe: int = 0, n_rg: int = 0,
          banks: bool = False, hyper: bool = False) -> int:
    blk = C * 9 + C + 2 * C * C + 2 * C + C * _hidden(C, block) + C
    return (C * 192 + C + C * 2 * C + C + n_enc * blk + C * C * 4 + C
            + 2 * C * C + 2 * C + 4 * C * C + 4 * C + C * 2 * C + C
            + n_dec * blk + 192 * C + 192
            + (n_fe + n_rg) * blk + (4 * NUM_QP * C if banks else 0)
            + (hyper_count(C) if hyper else 0))


def unpack(flat: np.ndarray, C: int, n_enc: int, n_dec: int, block: str = "lrelu", n_fe: int = 0,
           n_rg: int = 0, banks: bool = False, hyper: bool = False) -> Params:
    flat = np.asarray(flat, dtype=np.float64).reshape(-1)
    want = count(C, n_enc, n_dec, block, n_fe, n_rg, banks, hyper)
    if flat.size != want:
        raise ValueError(f"expected {want} parameters, got {flat.size}")
    pos = 0

    def take(shape):
        nonlocal pos
        n = int(np.prod(shape))
        v = flat[pos:pos + n].reshape(shape)
        pos += n
        return v

    def conv(wshape):
        w = take(wshape)
        b = take((wshape[0],))
        return Conv(w, b)

    def blk():
        return Block(conv((C, 3, 3)), conv((2 * C, C)), conv((C, _hidden(C, block))), block)

    pe = conv((C, 192))
    fuse_enc = conv((C, 2 * C))
    enc = [blk() for _ in range(n_enc)]
    down = conv((C, C, 2, 2))
    head = conv((2 * C, C))
    up = conv((4 * C, C))
    fuse_dec = conv((C, 2 * C))
    dec = [blk() for _ in range(n_dec)]
    rec = conv((192, C))
    fe = [blk() for _ in range(n_fe)]
    rg = [blk() for _ in range(n_rg)]
    bk = {name: take((NUM_QP, C)) for name in ("q_e", "q_d", "q_f", "q_r")} if banks else None
    hy = None
    if hyper:
        zana = conv((CZ, C, 2, 2))
        zsyn = conv((8 * C, CZ))
        step2 = conv((C, C // 2))
        hy = Hyper(zana, zsyn, step2, take((NUM_QP, CZ)))
    assert pos == flat.size
    return Params(C, pe, fuse_enc, enc, down, head, up, fuse_dec, dec, rec, block, fe, rg, bk, hy)


def _f16(v: np.ndarray) -> np.ndarray:
    return np.asarray(v, dtype=np.float64).astype(np.float16).astype(np.float64)


def bank_vectors(p: Params, qp) -> tuple:
    """The four bank vectors (q_e, q_d, q_f, q_r) at rate point qp in [0, 63].
    Integer qp: row qp.  Between two rate points the supplementary
    rate-adjustment section interpolates the vectors linearly; with
    i = min(floor(qp), 62) and t = qp - i the vector is (1 - t) row i +
    t row i+1 (float64; exactly row qp when qp is an integer)."""
    qp = float(qp)
    if not 0.0 <= qp <= NUM_QP - 1:
        raise ValueError(f"qp must be in [0, {NUM_QP - 1}]")
    i = min(int(np.floor(qp)), NUM_QP - 2)
    t = qp - i
    return tuple((1.0 - t) * p.banks[n][i] + t * p.banks[n][i + 1] for n in ("q_e", "q_d", "q_f", "q_r"))


def fold_qp(p: Params, qp) -> Params:
    """Params with the vector banks at rate point qp (:func:`bank_vectors`)
    folded into the convolutions next to them, each folded value rounded to
    fp16 once (the precision of every weight):
      q_e scales y:           down rows and bias,  W'[o] = q_e[o] W[o]
      q_d scales yhat:        up columns,          W'[:, c] = W[:, c] q_d[c]
      q_f scales the context: fuse columns C..2C,  W'[:, C + c] = W[:, C + c] q_f[c]
      q_r scales the rg output: rec columns,       W'[:, c] = W[:, c] q_r[c]
    Without banks, p itself."""
    if p.banks is None:
        return p
    C = p.C
    qe, qd, qf, qr = bank_vectors(p, qp)
    down = Conv(_f16(p.down.w * qe[:, None, None, None]), _f16(p.down.b * qe))
    up = Conv(_f16(p.up.w * qd[None, :]), p.up.b)

    def ctx_cols(c: Conv) -> Conv:
        w = np.array(c.w)
        w[:, C:] = _f16(w[:, C:] * qf[None, :])
        return Conv(w, c.b)

    rec = Conv(_f16(p.rec.w * qr[None, :]), p.rec.b)
    return dataclasses.replace(p, down=down, up=up, fuse_enc=ctx_cols(p.fuse_enc),
                               fuse_dec=ctx_cols(p.fuse_dec), rec=rec)
