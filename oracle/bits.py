"""Gaussian likelihood and bit estimate of the quantised latent.

The paper's entropy model predicts a distribution per latent element and
codes the rounded symbols (Fig. 4 "Q", Supp. B.2).  The transform studied
here uses a zero-mean Gaussian of scale sigma on the residual q = round(y - mu):

  L(q)  = Phi((q + 1/2) / sigma) - Phi((q - 1/2) / sigma)
        = 1/2 [erfc((|q| - 1/2) / (sigma sqrt 2)) - erfc((|q| + 1/2) / (sigma sqrt 2))]
  bits  = sum over elements of -log2(max(L, 1e-9))

The second line is the same quantity written with upper tails (symmetric in
q), which avoids cancellation for large |q|.  sigma = max(softplus(s), 0.11).
"""
from __future__ import annotations

import numpy as np
from scipy.special import erfc

SIGMA_MIN = 0.11
L_MIN = 1e-9


def softplus(s: np.ndarray) -> np.ndarray:
    s = np.asarray(s, dtype=np.float64)
    return np.where(s > 30.0, s, np.log1p(np.exp(np.minimum(s, 30.0))))


def sigma_from_s(s: np.ndarray) -> np.ndarray:
    return np.maximum(softplus(s), SIGMA_MIN)


def likelihood(q: np.ndarray, sigma: np.ndarray) -> np.ndarray:
    a = np.abs(np.asarray(q, dtype=np.float64))
    sg = np.asarray(sigma, dtype=np.float64) * np.sqrt(2.0)
    return 0.5 * (erfc((a - 0.5) / sg) - erfc((a + 0.5) / sg))


def element_bits(q: np.ndarray, sigma: np.ndarray) -> np.ndarray:
    return -np.log2(np.maximum(likelihood(q, sigma), L_MIN))


def estimate_bits(q: np.ndarray, sigma: np.ndarray) -> float:
    """Total estimated bits of the symbols q under Gaussian(0, sigma)."""
    return float(np.sum(element_bits(q, sigma)))
