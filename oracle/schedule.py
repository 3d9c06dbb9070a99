"""Noise schedule and time grid (test infrastructure only).

Background, eq. (interpolating-forward): alpha_t decreases monotonically from
alpha_0 = 1 (clean data) to alpha_1 = 0 (the prior).  The workloads use the
linear schedule alpha_t = 1 - t.  The paper does not state the time grid; this
build reads it as t_k = k / T, k = T .. 1, so step k maps z_{t_k} to
z_{t_{k-1}} with (alpha_t, alpha_s) = (alpha(k/T), alpha((k-1)/T)), and the last
step has alpha_s = alpha_0 = 1.

Pinned: alpha_0 = 1, alpha_1 = 0, strictly decreasing (tests).
"""
import numpy as np


def alpha(t):
    return 1.0 - np.asarray(t, dtype=np.float64)


def alphas(T):
    """alphas[k] = alpha(k / T) for k = 0..T (float64)."""
    k = np.arange(T + 1, dtype=np.float64)
    return alpha(k / T)


def alpha_t_given_s(alpha_t, alpha_s):
    """alpha_{t|s}, the schedule of the transition q(z_t | z_s).

    The paper uses alpha_{t|s} in eq. (uniform_true_reverse_posterior) without
    restating it; composing q(z_s | x) with q(z_t | z_s), both of the
    interpolating form, must give q(z_t | x), which forces
    alpha_t = alpha_{t|s} * alpha_s.  Pinned by the brute-force composition test.
    """
    return alpha_t / alpha_s
