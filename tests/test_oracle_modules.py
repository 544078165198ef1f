"""Pins of the conditional-coding modules in the oracle (Fig. 4; Sec. 4.3, 4.4):
feature extractor (context F_{t-1} from f_{t-1}), reconstruction generation,
and the qp-indexed vector banks folded into the adjacent convolutions.

* The parameter count against the synthetic list, shapes, rejection of a
  wrong length.
* fold_qp against a per-element restatement, the identity for all-one banks,
  the range check.
* The whole float transform with both modules against an independent
  re-implementation from torch convolutions.
* Int path: encoder and decoder states agree frame after frame.
* Rate control: with the synthetic banks, the estimated bits fall as qp rises.
"""
import dataclasses

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth
from oracle import codec_float as cf
from oracle import codec_int as ci
from oracle import params as P


def t64(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))


def modular(C=64, ne=2, nd=2, nfe=2, nrg=1, banks=True, block="lrelu"):
    flat = synth.make_weights(C, ne, nd, block=block, n_fe=nfe, n_rg=nrg, banks=banks)
    return flat, oracle.unpack(flat, C, ne, nd, block=block, n_fe=nfe, n_rg=nrg, banks=banks)


def test_count_shapes_and_length_check():
    for C in (64, 256):
        n = sum(int(np.prod(s)) for _, s, _, _ in synth.param_list(C, 2, 3, "lrelu", 4, 1, True))
        assert n == P.count(C, 2, 3, "lrelu", 4, 1, True)
        assert n - P.count(C, 2, 3) == 5 * (P.count(C, 1, 0) - P.count(C, 0, 0)) + 4 * 64 * C
    flat, p = modular()
    assert len(p.fe) == 2 and len(p.rg) == 1 and set(p.banks) == {"q_e", "q_d", "q_f", "q_r"}
    assert all(v.shape == (64, 64) for v in p.banks.values())
    with pytest.raises(ValueError):
        oracle.unpack(flat[:-1], 64, 2, 2, n_fe=2, n_rg=1, banks=True)


def test_fold_qp_restated_per_element():
    _, p = modular(C=64, ne=1, nd=1, nfe=0, nrg=0)
    qp = 37
    f = P.fold_qp(p, qp)
    qe, qd, qf, qr = (p.banks[n][qp] for n in ("q_e", "q_d", "q_f", "q_r"))
    r16 = lambda v: float(np.float16(v))  # noqa: E731
    rng = np.random.default_rng(0)
    for _ in range(200):
        o, c, i, j = rng.integers(0, 64, 4) % [64, 64, 2, 2]
        assert f.down.w[o, c, i, j] == r16(p.down.w[o, c, i, j] * qe[o])
        assert f.down.b[o] == r16(p.down.b[o] * qe[o])
        n, k = rng.integers(0, 256), rng.integers(0, 64)
        assert f.up.w[n, k] == r16(p.up.w[n, k] * qd[k])
        n, k = rng.integers(0, 64), rng.integers(0, 128)
        want = r16(p.fuse_enc.w[n, k] * qf[k - 64]) if k >= 64 else p.fuse_enc.w[n, k]
        assert f.fuse_enc.w[n, k] == want
        want = r16(p.fuse_dec.w[n, k] * qf[k - 64]) if k >= 64 else p.fuse_dec.w[n, k]
        assert f.fuse_dec.w[n, k] == want
        n, k = rng.integers(0, 192), rng.integers(0, 64)
        assert f.rec.w[n, k] == r16(p.rec.w[n, k] * qr[k])
    np.testing.assert_array_equal(f.up.b, p.up.b)
    np.testing.assert_array_equal(f.head.w, p.head.w)
    with pytest.raises(ValueError):
        P.fold_qp(p, 64)


def test_fold_qp_with_unit_banks_is_the_identity():
    _, p = modular(C=64, ne=1, nd=1, nfe=0, nrg=0)
    ones = {k: np.ones_like(v) for k, v in p.banks.items()}
    f = P.fold_qp(dataclasses.replace(p, banks=ones), 5)
    for name in ("down", "up", "fuse_enc", "fuse_dec", "rec"):
        np.testing.assert_array_equal(getattr(f, name).w, getattr(p, name).w)
        np.testing.assert_array_equal(getattr(f, name).b, getattr(p, name).b)
    _, p0 = modular(C=64, ne=1, nd=1, nfe=0, nrg=0, banks=False)
    assert P.fold_qp(p0, 5) is p0


def torch_block(z, blk):
    C = z.shape[1]
    a = F.conv2d(z, t64(blk.dw.w)[:, None], t64(blk.dw.b), padding=1, groups=C)
    h = F.conv2d(a, t64(blk.pw1.w)[:, :, None, None], t64(blk.pw1.b))
    return z + F.conv2d(F.leaky_relu(h, 0.1), t64(blk.pw2.w)[:, :, None, None], t64(blk.pw2.b))


def test_transform_with_modules_matches_torch():
    _, p = modular()
    pq = P.fold_qp(p, 20)
    x = synth.random_frame(64, 64, seed=3)
    rng = np.random.default_rng(1)
    f_prev = rng.standard_normal((64, 8, 8)) * 0.5
    # torch: context by the extractor's blocks, encoder, reconstruction generation
    ctx = t64(f_prev)[None]
    for blk in pq.fe:
        ctx = torch_block(ctx, blk)
    e = F.conv2d(t64(x)[None], t64(pq.pe.w.reshape(64, 3, 8, 8)), t64(pq.pe.b), stride=8)
    z = F.conv2d(torch.cat([e, ctx], 1), t64(pq.fuse_enc.w)[:, :, None, None], t64(pq.fuse_enc.b))
    for blk in pq.enc:
        z = torch_block(z, blk)
    y = F.conv2d(z, t64(pq.down.w), t64(pq.down.b), stride=2)
    np.testing.assert_allclose(cf.analysis(pq, x, f_prev), y[0].numpy(), rtol=1e-10, atol=1e-10)
    r = t64(f_prev)[None]
    for blk in pq.rg:
        r = torch_block(r, blk)
    wr = t64(pq.rec.w.reshape(3, 8, 8, 64).transpose(3, 0, 1, 2))
    xr = F.conv_transpose2d(r, wr, None, stride=8)
    xr = torch.clamp(xr + t64(pq.rec.b.reshape(3, 8, 8)).repeat(1, 8, 8)[None], 0, 1)
    np.testing.assert_allclose(cf.reconstruct(pq, f_prev), xr[0].numpy(), rtol=1e-10, atol=1e-10)


def test_int_states_agree_with_modules():
    _, p = modular()
    ip = ci.integerize(P.fold_qp(p, 40))
    se = ci.zero_state(ip, 64, 64)
    sd = ci.zero_state(ip, 64, 64)
    for x in synth.frame_sequence("tiny", 2):
        r = ci.encode_frame(ip, x, se)
        xhat, sd = ci.decode_frame(ip, r.q, sd)
        np.testing.assert_array_equal(sd.feat, r.state.feat)
        np.testing.assert_array_equal(sd.yhat, r.state.yhat)
        assert 0 <= xhat.min() and xhat.max() <= 512
        se = r.state


def test_bits_fall_as_qp_rises():
    _, p = modular(nfe=1, nrg=0)
    x = synth.random_frame(64, 64, seed=8)
    bits = []
    for qp in (0, 32, 63):
        pq = P.fold_qp(p, qp)
        r = cf.encode_frame(pq, x, cf.zero_state(pq, 64, 64))
        bits.append(r.bits)
    assert bits[0] > bits[1] > bits[2], bits


def test_bank_vectors_between_rate_points():
    _, p = modular(C=64, ne=1, nd=1, nfe=0, nrg=0)
    names = ("q_e", "q_d", "q_f", "q_r")
    for qp in range(64):  # the learned points themselves, exactly
        for v, n in zip(P.bank_vectors(p, qp), names):
            np.testing.assert_array_equal(v, p.banks[n][qp])
    for i in (0, 17, 62):
        lo, hi = p.banks["q_d"][i], p.banks["q_d"][i + 1]
        mid = P.bank_vectors(p, i + 0.5)[1]
        np.testing.assert_allclose(mid, 0.5 * (lo + hi), rtol=0, atol=1e-15)
        # on the segment between the two points, at a quarter of the way
        q1 = P.bank_vectors(p, i + 0.25)[1]
        np.testing.assert_allclose(q1 - lo, 0.25 * (hi - lo), rtol=0, atol=1e-15)
        assert np.all(np.minimum(lo, hi) - 1e-15 <= q1) and np.all(q1 <= np.maximum(lo, hi) + 1e-15)
    for bad in (-0.25, 63.5, float("nan")):
        with pytest.raises(ValueError):
            P.bank_vectors(p, bad)
    # the fold at an interpolated rate differs from both neighbours
    f = P.fold_qp(p, 20.5)
    assert not np.array_equal(f.up.w, P.fold_qp(p, 20).up.w)
    assert not np.array_equal(f.up.w, P.fold_qp(p, 21).up.w)


def test_bits_at_an_interpolated_rate_lie_between():
    _, p = modular(nfe=1, nrg=0)
    x = synth.random_frame(64, 64, seed=8)
    bits = []
    for qp in (0, 31.5, 63):
        pq = P.fold_qp(p, qp)
        bits.append(cf.encode_frame(pq, x, cf.zero_state(pq, 64, 64)).bits)
    assert bits[0] > bits[1] > bits[2], bits
