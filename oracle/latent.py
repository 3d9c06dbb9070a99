"""Gaussian-latent argmax projection (test infrastructure only).

App. A.5 (Discrete Consistency Distillation): uniform-state discrete diffusion
is the argmax projection of a Gaussian diffusion on the one-hot vectors.  For
one position with clean token x the discrete latent is

  z = argmax_v ( alpha_tilde [v == x] + sigma eps_v ),  eps ~ N(0, I_V),
  alpha_tilde**2 + sigma**2 = 1,

eps_v = N(word(STREAM_LATENT, step, row, v)) (noise.normal_icdf); the lowest
index wins a tie.

The paper does not print the map between alpha_tilde and the discrete
schedule alpha.  Reading adopted here: z = x exactly when every other latent
falls below alpha_tilde / sigma + eps_x, so

  P(z = x) = integral phi(u) Phi(u + alpha_tilde / sigma)**(K - 1) du,

and, z being uniform over the other K - 1 classes otherwise, matching the
interpolating forward process Cat(alpha x + (1 - alpha) 1/K) requires
alpha = (K P(z = x) - 1) / (K - 1).  `alpha_of_tilde` evaluates this by
trapezoidal quadrature; `tilde_of_alpha` inverts it by bisection.

Pinned by Monte-Carlo frequencies of `latent_argmax` against the quadrature
(binomial test), uniformity of the non-x outcomes (chi-square) and
alpha_tilde = 0 giving a uniform token.
"""
import numpy as np
from scipy.special import log_ndtr

from . import noise as _nz
from . import philox as _ph


def latent_argmax(x, V, alpha_tilde, sigma, seed, step, rows=None):
    """z [R] for clean tokens x [R], evaluated with all V latents per position."""
    x = np.asarray(x)
    rows = np.arange(x.shape[0]) if rows is None else np.asarray(rows)
    out = np.empty(x.shape[0], dtype=np.int64)
    v = np.arange(V)
    for i in range(x.shape[0]):
        eps = _nz.normal_icdf(_ph.counter_words(seed, _ph.STREAM_LATENT, step, int(rows[i]), v))
        score = sigma * eps
        score[int(x[i])] += alpha_tilde
        out[i] = int(np.argmax(score))
    return out


def p_keep(alpha_tilde, K, n=40001, lim=14.0):
    """P(z = x) for K classes at latent signal level alpha_tilde in [0, 1)."""
    sigma = np.sqrt(1.0 - alpha_tilde ** 2)
    u = np.linspace(-lim, lim, n)
    log_phi = -0.5 * u * u - 0.5 * np.log(2.0 * np.pi)
    f = np.exp(log_phi + (K - 1) * log_ndtr(u + alpha_tilde / sigma))
    return float(np.trapezoid(f, u))


def alpha_of_tilde(alpha_tilde, K):
    return (K * p_keep(alpha_tilde, K) - 1.0) / (K - 1.0)


def tilde_of_alpha(alpha, K, tol=1e-12):
    """alpha_tilde in [0, 1) whose argmax projection has discrete schedule value alpha."""
    if alpha <= 0.0:
        return 0.0
    lo, hi = 0.0, 1.0 - 1e-12
    while hi - lo > tol:
        mid = 0.5 * (lo + hi)
        if alpha_of_tilde(mid, K) < alpha:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)
