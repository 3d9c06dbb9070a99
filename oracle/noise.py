"""Transforms of a uniform 32-bit word into the noise the sampler uses
(test infrastructure only).

The paper does not specify how uniforms, Gumbels or normals are produced; the
definitions below are the reading adopted here, chosen so that every value is
exactly defined in float64:

  u(w)  = (w + 1/2) * 2**-32                 in (0, 1), exact in float64
  c(w)  = 1 - u(w) = (2**32 - 1 - w + 1/2) * 2**-32, exact
  E(w)  = -log u(w)  (evaluated as -log1p(-c) when u >= 1/2)  ~ Exp(1)
  G(w)  = -log E(w)                                          ~ Gumbel(0, 1)
  N(w)  = Phi^-1(u(w))  (evaluated as -Phi^-1(c) when u >= 1/2)  ~ N(0, 1)

Parameter initialisation uses Box-Muller on a pair of words (u1, u2):
  r = sqrt(-2 log u1); even element r cos(2 pi u2), odd element r sin(2 pi u2).

Pinned by Kolmogorov-Smirnov tests against the exact distributions and by the
exact-value checks in the oracle self-tests.
"""
import numpy as np
from scipy.special import ndtri

_TWO_M32 = 2.0 ** -32


def uniform(w):
    w = np.asarray(w, dtype=np.float64)
    return (w + 0.5) * _TWO_M32


def complement(w):
    w = np.asarray(w, dtype=np.float64)
    return (4294967295.0 - w + 0.5) * _TWO_M32


def exponential(w):
    """E = -log u with full relative accuracy for u close to 1."""
    w = np.asarray(w, dtype=np.uint32)
    u = uniform(w)
    c = complement(w)
    hi = w >= np.uint32(2 ** 31)
    with np.errstate(divide="ignore"):
        return np.where(hi, -np.log1p(-c), -np.log(u))


def gumbel(w):
    return -np.log(exponential(w))


def normal_icdf(w):
    """Standard normal by inversion of the CDF (monotone increasing in w)."""
    w = np.asarray(w, dtype=np.uint32)
    u = uniform(w)
    c = complement(w)
    hi = w >= np.uint32(2 ** 31)
    return np.where(hi, -ndtri(c), ndtri(u))


def box_muller(w1, w2, odd):
    """Box-Muller normal from two words; `odd` selects the sine branch."""
    u1 = uniform(w1)
    u2 = uniform(w2)
    r = np.sqrt(-2.0 * np.log(u1))
    ang = 2.0 * np.pi * u2
    return np.where(np.asarray(odd, dtype=bool), r * np.sin(ang), r * np.cos(ang))
