"""Pins for the likelihood / bit estimate: closed forms, library CDF, normalisation."""
import math

import numpy as np
import pytest
from scipy.special import erf
from scipy.stats import norm

from oracle import bits


@pytest.mark.parametrize("sigma", [0.11, 0.3, 1.0, 2.5, 17.0])
def test_likelihood_matches_normal_cdf_difference(sigma):
    q = np.arange(-6, 7)
    ref = norm.cdf((q + 0.5) / sigma) - norm.cdf((q - 0.5) / sigma)
    np.testing.assert_allclose(bits.likelihood(q, np.full(q.shape, sigma)), ref, rtol=1e-9, atol=1e-15)


@pytest.mark.parametrize("sigma", [0.11, 0.7, 3.0, 40.0])
def test_likelihood_telescopes_to_one(sigma):
    # sum_{q=-M..M} L(q) = erf((M + 1/2) / (sigma sqrt 2)) exactly (telescoping CDF differences)
    for M in (0, 1, 5, 50):
        q = np.arange(-M, M + 1)
        s = bits.likelihood(q, np.full(q.shape, sigma)).sum()
        assert abs(s - erf((M + 0.5) / (sigma * math.sqrt(2)))) < 1e-12
    q = np.arange(-2000, 2001)
    assert abs(bits.likelihood(q, np.full(q.shape, sigma)).sum() - 1.0) < 1e-12


def test_likelihood_zero_symbol_and_symmetry():
    sig = np.array([0.2, 1.0, 5.0])
    np.testing.assert_allclose(bits.likelihood(np.zeros(3), sig), erf(1.0 / (2 * math.sqrt(2) * sig)), rtol=1e-14)
    q = np.array([1, 2, 7, 30])
    s = np.full(4, 1.3)
    np.testing.assert_array_equal(bits.likelihood(q, s), bits.likelihood(-q, s))


def test_tail_has_no_cancellation():
    # far tail: upper-tail form keeps full relative precision where CDF differences underflow to 0
    q, sigma = 12.0, 1.0
    L = bits.likelihood(np.array([q]), np.array([sigma]))[0]
    ref = norm.sf((q - 0.5) / sigma) - norm.sf((q + 0.5) / sigma)
    assert L > 0 and abs(L / ref - 1) < 1e-10


def test_bits_floor_and_total():
    # L clamped at 1e-9 -> at most -log2(1e-9) bits per element
    b = bits.element_bits(np.array([1000]), np.array([0.11]))
    assert b[0] == pytest.approx(-math.log2(1e-9), rel=1e-15)
    q = np.array([0, 1, -1, 3])
    s = np.array([1.0, 1.0, 1.0, 2.0])
    ref = sum(-math.log2(norm.cdf((qq + .5) / ss) - norm.cdf((qq - .5) / ss)) for qq, ss in zip(q, s))
    assert bits.estimate_bits(q, s) == pytest.approx(ref, rel=1e-12)


def test_sigma_mapping():
    s = np.array([-50.0, -3.0, 0.0, 2.0, 40.0, 100.0])
    sg = bits.sigma_from_s(s)
    ref = np.maximum(np.log1p(np.exp(np.minimum(s, 700))), 0.11)
    np.testing.assert_allclose(sg, ref, rtol=1e-15)
    assert sg[0] == 0.11 and sg[2] == pytest.approx(math.log(2.0))
