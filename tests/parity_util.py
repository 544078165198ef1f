"""Helpers shared by the GPU parity tests (comparison rules and crops)."""
from __future__ import annotations

import numpy as np

import oracle
import synth
from oracle import codec_float as cf
from oracle import codec_int as ci

FP16_TOL = 2e-2  # |gpu - ref| <= 2e-2 * max(1, |ref|) on the fp16 path


def assert_close_fp16(got, ref, what, tol=FP16_TOL):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    err = np.abs(got - ref)
    lim = tol * np.maximum(1.0, np.abs(ref))
    bad = err > lim
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} elements out of tolerance, "
                           f"max err {err.max():.4g} (at ref {ref.flat[int(np.argmax(err))]:.4g})")
    return float(err.max())


def q_band(y, mu, tol=FP16_TOL):
    """Elements whose rounding y - mu is ambiguous within the fp16 error band."""
    d = np.asarray(y, np.float64) - np.asarray(mu, np.float64)
    frac = d - np.floor(d)
    return np.abs(frac - 0.5) <= tol * np.maximum(1.0, np.abs(np.asarray(y, np.float64)))


def params_for(C, ne, nd, block="lrelu"):
    flat = synth.make_weights(C, ne, nd, block=block)
    p = oracle.unpack(flat, C, ne, nd, block=block)
    return flat, p


def check_fp16_encode(p, x, feat_prev, yhat_prev, q_gpu, bits_gpu, feat_new, yhat_new, what="",
                      valid=None):
    """Teacher-forced fp16 comparison of one encoded frame.

    The oracle starts from the GPU's state; q must agree outside the rounding
    band; bits, yhat and f_t are compared using the GPU's q.  ``valid`` is an
    optional (latent-grid slice, 1/8-grid slice) pair restricting the
    comparison to a region (crops)."""
    y = cf.analysis(p, x, feat_prev)
    mu, s = cf.prior(p, yhat_prev)
    q = np.asarray(q_gpu, np.float64)
    band = q_band(y, mu)
    q_ref = np.rint(y - mu)
    sl16, sl8 = valid if valid is not None else (np.s_[:, :, :], np.s_[:, :, :])
    mism = (q != q_ref) & ~band
    assert not mism[sl16].any(), f"{what}: q differs outside the rounding band at {int(mism[sl16].sum())} elements"
    far = np.abs(q - q_ref) > 1
    assert not far[sl16].any(), f"{what}: q off by more than 1 inside the rounding band at {int(far[sl16].sum())} elements"
    # reading A16 allows a flip only inside the band; as a guard against a
    # systematic shift, at most 1 % of the symbols may flip (2 where that is
    # fewer: one latent pixel has only C symbols, a few of them in the band)
    flips = int(np.count_nonzero((q != q_ref)[sl16]))
    n = int(np.asarray(q[sl16]).size)
    assert flips <= max(2, 0.01 * n), f"{what}: {flips} of {n} symbols flipped inside the rounding band"
    yhat_ref = q + mu
    assert_close_fp16(np.asarray(yhat_new)[sl16], yhat_ref[sl16], what + " yhat")
    f_ref = cf.decoder_feature(p, yhat_ref, feat_prev)
    err = assert_close_fp16(np.asarray(feat_new)[sl8], f_ref[sl8], what + " f_t")
    if bits_gpu is not None:
        ref_bits = oracle.estimate_bits(q[sl16], oracle.sigma_from_s(s)[sl16])
        assert abs(bits_gpu - ref_bits) <= 1e-2 * abs(ref_bits), (what, bits_gpu, ref_bits)
    return f_ref, err


def int_state(feat, yhat):
    return ci.State(np.asarray(feat, np.int64), np.asarray(yhat, np.int64))
