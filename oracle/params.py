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


def _hidden(C: int, block: str) -> int:
    if block not in ("lrelu", "gated"):
        raise ValueError(f"unknown block form {block!r}")
    return 2 * C if block == "lrelu" else C


def count(C: int, n_enc: int, n_dec: int, block: str = "lrelu") -> int:
    blk = C * 9 + C + 2 * C * C + 2 * C + C * _hidden(C, block) + C
    return (C * 192 + C + C * 2 * C + C + n_enc * blk + C * C * 4 + C
            + 2 * C * C + 2 * C + 4 * C * C + 4 * C + C * 2 * C + C
            + n_dec * blk + 192 * C + 192)


def unpack(flat: np.ndarray, C: int, n_enc: int, n_dec: int, block: str = "lrelu") -> Params:
    flat = np.asarray(flat, dtype=np.float64).reshape(-1)
    if flat.size != count(C, n_enc, n_dec, block):
        raise ValueError(f"expected {count(C, n_enc, n_dec, block)} parameters, got {flat.size}")
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
    assert pos == flat.size
    return Params(C, pe, fuse_enc, enc, down, head, up, fuse_dec, dec, rec, block)
