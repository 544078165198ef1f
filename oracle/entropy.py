"""Entropy coding of the quantised latent: quantised-scale Gaussian tables and
interleaved rANS.  TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper codes the symbols q = RHE(y - mu) with an arithmetic coder driven by
the entropy model's distribution (Fig. 4 "AE"/"AD", Fig. 6 and Supp. B.2), and
the integer path exists so that encoder and decoder derive the same
distribution on any device (Sec. 4.5).  This module is the plain reference of
the coder the library implements on the GPU.  Everything here is a fixed
format; the numbers below are its definition, not tuning knobs.

Distribution tables (one per scale index j = 0 .. NS-1):
  sigma_j  = float32(SMIN * (SMAX / SMIN) ** (j / (NS - 1)))
  R_j      = max(ceil(TAIL * sigma_j), RMIN)
  symbols  q = -R_j .. R_j, then ESC (|q| > R_j)
  p(q)     = 1/2 [erfc((|q| - 1/2) / (sigma_j sqrt2)) - erfc((|q| + 1/2) / (sigma_j sqrt2))]
  p(ESC)   = erfc((R_j + 1/2) / (sigma_j sqrt2))
  f        = 1 + floor(p * (M - n)) for each of the n = 2 R_j + 2 symbols,
             and the remainder M - sum(f) added to f(q = 0); M = 2^16.
  The scale index of a sigma is the smallest j with sigma_j >= sigma (NS - 1
  if there is none).

rANS (Duda, "Asymmetric numeral systems", 2013; the range variant with a
32-bit state x in [L, 2^32), L = 2^16, and 16-bit renormalisation words):
  encode (s with start c, frequency f):
      if x >= f * 2^16: emit x mod 2^16, x = x div 2^16
      x = (x div f) * M + (x mod f) + c
  decode: slot = x mod M; s = the symbol with c <= slot < c + f;
      x = f * (x div M) + slot - c;  if x < L: x = x * 2^16 + next word.
  The encoder runs over the symbols in reverse; its words, read backwards,
  are the decoder's input.  Each state starts at L and ends as two words.

An escaped symbol continues with one uniform sub-symbol of frequency 1 (a
plain 16-bit field): 32768 * sign + v with v = |q| - R_j - 1 (v < 32768
because |q| <= 32768 and R_j >= 32).

Streams: the symbols are cut into streams of LANES * STEPS; inside a stream,
symbol i belongs to lane i mod LANES at step i div LANES, and the LANES lanes
each run their own rANS state in lock step.  At every (step, sub-symbol) the
lanes that read a word read the next words of the stream in increasing lane
order; the stream opens with the LANES initial states (two words each, high
half first, lane order).  A partial last stream has fewer symbols (lanes and
steps past the end take part in nothing, but every lane keeps its state).

Container (little-endian): u32 magic 'NCRS', u32 version 1, u32 number of
symbols, u32 symbols per stream, u32 number of streams, u16 length of each
stream in words, zero padding to a multiple of 4 bytes, then the streams'
words back to back.
"""
from __future__ import annotations

import math
import struct

import numpy as np
from scipy.special import erfc

NS = 64
SMIN = 0.11
SMAX = 256.0
TAIL = 8.0
RMIN = 32
PREC = 16
M = 1 << PREC
L = 1 << 16
LANES = 64
STEPS = 128
STREAM = LANES * STEPS
MAGIC = 0x5352434E  # 'N', 'C', 'R', 'S'
VERSION = 1


def scale_table() -> np.ndarray:
    """sigma_j, j = 0 .. NS-1, as float32."""
    j = np.arange(NS, dtype=np.float64)
    return (SMIN * (SMAX / SMIN) ** (j / (NS - 1))).astype(np.float32)


def scale_index(sigma) -> np.ndarray:
    """Smallest j with sigma_j >= sigma, else NS - 1 (compared in float64)."""
    tab = scale_table().astype(np.float64)
    s = np.asarray(sigma, dtype=np.float64)
    k = np.searchsorted(tab, s, side="left")
    return np.minimum(k, NS - 1).astype(np.int64)


def table(j: int):
    """(R, freq, start) of scale j; entries are q = -R .. R then ESC."""
    sigma = float(scale_table()[j])
    R = max(int(math.ceil(TAIL * sigma)), RMIN)
    n = 2 * R + 2
    sg = sigma * math.sqrt(2.0)
    a = np.abs(np.arange(-R, R + 1, dtype=np.float64))
    p = np.empty(n, dtype=np.float64)
    p[:-1] = 0.5 * (erfc((a - 0.5) / sg) - erfc((a + 0.5) / sg))
    p[-1] = erfc((R + 0.5) / sg)
    f = 1 + np.floor(p * (M - n)).astype(np.int64)
    f[R] += M - int(f.sum())
    start = np.concatenate([[0], np.cumsum(f)[:-1]]).astype(np.int64)
    return R, f, start


_TABLES = None


def tables():
    global _TABLES
    if _TABLES is None:
        _TABLES = [table(j) for j in range(NS)]
    return _TABLES


def _subsymbols(q: int, j: int):
    """The (start, freq) sub-symbols of one symbol, in decoding order."""
    R, f, c = tables()[j]
    if -R <= q <= R:
        return [(int(c[q + R]), int(f[q + R]))]
    v = abs(q) - R - 1
    return [(int(c[-1]), int(f[-1])), ((32768 if q < 0 else 0) + v, 1)]


def encode_stream(q: np.ndarray, k: np.ndarray) -> list:
    """Words (decoding order) of one stream of len(q) <= STREAM symbols."""
    n = len(q)
    steps = (n + LANES - 1) // LANES
    subs = [[None] * LANES for _ in range(steps)]
    for i in range(n):
        subs[i // LANES][i % LANES] = _subsymbols(int(q[i]), int(k[i]))
    x = [L] * LANES
    rev = []  # groups of words, each group in increasing lane order, groups in reverse decoding order
    for t in range(steps - 1, -1, -1):
        nsub = max(len(s) for s in subs[t] if s is not None)
        for u in range(nsub - 1, -1, -1):
            group = []
            for lane in range(LANES):
                s = subs[t][lane]
                if s is None or u >= len(s):
                    continue
                c, f = s[u]
                if x[lane] >= f << 16:
                    group.append(x[lane] & 0xFFFF)
                    x[lane] >>= 16
                x[lane] = (x[lane] // f) * M + (x[lane] % f) + c
            rev.append(group)
    words = []
    for lane in range(LANES):
        words += [x[lane] >> 16, x[lane] & 0xFFFF]
    for group in reversed(rev):
        words += group
    return words


def _find(j: int, slot: int) -> int:
    R, f, c = tables()[j]
    return int(np.searchsorted(c, slot, side="right") - 1)


def decode_stream(words, k: np.ndarray):
    """Symbols of one stream (len(k) of them) and whether the words were
    consumed exactly with every state back at L."""
    n = len(k)
    steps = (n + LANES - 1) // LANES
    if len(words) < 2 * LANES:
        return np.zeros(n, dtype=np.int64), False
    x = [(words[2 * ln] << 16) | words[2 * ln + 1] for ln in range(LANES)]
    pos = 2 * LANES
    ok = True
    out = np.zeros(n, dtype=np.int64)

    def take(slot_state, lane, c, f):
        nonlocal pos, ok
        xs = f * (slot_state >> PREC) + (slot_state & (M - 1)) - c
        if xs < L:
            if pos < len(words):
                xs = (xs << 16) | words[pos]
            else:
                ok = False
            pos += 1
        return xs

    for t in range(steps):
        lanes = [ln for ln in range(LANES) if t * LANES + ln < n]
        # main symbol
        esc = {}
        for ln in lanes:
            j = int(k[t * LANES + ln])
            R, f, c = tables()[j]
            i = _find(j, x[ln] & (M - 1))
            x[ln] = take(x[ln], ln, int(c[i]), int(f[i]))
            if i == 2 * R + 1:
                esc[ln] = R
            else:
                out[t * LANES + ln] = i - R
        # escaped symbols: one 16-bit field each, lanes in order
        for ln in sorted(esc):
            fld = x[ln] & (M - 1)
            x[ln] = take(x[ln], ln, fld, 1)
            mag = esc[ln] + 1 + (fld & 32767)
            out[t * LANES + ln] = -mag if fld >= 32768 else mag
    ok = ok and pos == len(words) and all(v == L for v in x)
    return out, ok


def encode(q, k) -> bytes:
    """Container of the symbols q (int16 values) with scale indices k."""
    q = np.asarray(q, dtype=np.int64).ravel()
    k = np.asarray(k, dtype=np.int64).ravel()
    n = len(q)
    ns = (n + STREAM - 1) // STREAM
    streams = [encode_stream(q[i * STREAM:(i + 1) * STREAM], k[i * STREAM:(i + 1) * STREAM]) for i in range(ns)]
    head = struct.pack("<5I", MAGIC, VERSION, n, STREAM, ns)
    lens = struct.pack(f"<{ns}H", *[len(s) for s in streams])
    pad = b"\0" * ((-len(lens)) % 4)
    body = b"".join(struct.pack(f"<{len(s)}H", *s) for s in streams)
    return head + lens + pad + body


def decode(data: bytes, k):
    """(q, ok): the symbols of a container and whether it decoded cleanly."""
    k = np.asarray(k, dtype=np.int64).ravel()
    n = len(k)
    if len(data) < 20:
        return np.zeros(n, dtype=np.int64), False
    magic, ver, nsym, slen, ns = struct.unpack_from("<5I", data, 0)
    if magic != MAGIC or ver != VERSION or nsym != n or slen != STREAM or ns != (n + STREAM - 1) // STREAM:
        return np.zeros(n, dtype=np.int64), False
    lens = struct.unpack_from(f"<{ns}H", data, 20)
    off = 20 + 2 * ns + ((-2 * ns) % 4)
    if off + 2 * sum(lens) > len(data):
        return np.zeros(n, dtype=np.int64), False
    out = np.zeros(n, dtype=np.int64)
    ok = True
    for i in range(ns):
        w = list(struct.unpack_from(f"<{lens[i]}H", data, off))
        off += 2 * lens[i]
        qi, oki = decode_stream(w, k[i * STREAM:(i + 1) * STREAM])
        out[i * STREAM:i * STREAM + len(qi)] = qi
        ok = ok and oki
    return out, ok


def ideal_bits(q, k) -> float:
    """Sum of -log2(f / M) over all sub-symbols: the rANS payload up to the
    per-state flush."""
    total = 0.0
    for qi, ki in zip(np.asarray(q).ravel(), np.asarray(k).ravel()):
        for _, f in _subsymbols(int(qi), int(ki)):
            total += PREC - math.log2(f)
    return total
