"""Brute-force reverse posteriors by Bayes' rule over the forward process
(test infrastructure only; a pin of posterior.py).

Built only from Background, eq. (interpolating-forward): one step of the
forward process moves a one-hot state a to Cat(alpha a + (1 - alpha) pi), so
its transition matrix is Q(alpha)[a, b] = alpha [a == b] + (1 - alpha) pi_b.
With q(z_s | x) = Q(alpha_s)[x] and q(z_t | z_s) = Q(alpha_{t|s})[z_s], the
reverse posterior given a distribution x_theta over the clean token is

  p(z_s | z_t) = sum_x x_theta(x) q(z_s | x) q(z_t | z_s)
                 / sum_{x, z_s} x_theta(x) q(z_s | x) q(z_t | z_s)

(App. A.1 and A.2 state that the closed forms follow from Bayes' rule).
Everything is enumerated explicitly; nothing here uses the closed forms.
"""
import itertools

import numpy as np


def prior_vector(prior, V):
    """pi over K classes: the mask one-hot (K = V + 1) or uniform 1/K (K = V)."""
    if prior == "mask":
        pi = np.zeros(V + 1)
        pi[V] = 1.0
        return pi
    return np.full(V, 1.0 / V)


def transition(alpha, pi):
    K = pi.shape[0]
    return alpha * np.eye(K) + (1.0 - alpha) * np.tile(pi, (K, 1))


def posterior_bruteforce(prior, x, z_t, alpha_t, alpha_s):
    """Posterior over K classes for one position by explicit summation.

    Returns None when z_t has probability zero under the forward process
    (e.g. an unmasked token at alpha_t = 0), where no posterior exists."""
    x = np.asarray(x, dtype=np.float64)
    V = x.shape[0]
    pi = prior_vector(prior, V)
    K = pi.shape[0]
    Qs = transition(alpha_s, pi)
    Qts = transition(alpha_t / alpha_s, pi)
    px = np.zeros(K)
    px[:V] = x                      # clean data never holds the mask class
    num = np.zeros(K)
    for xc in range(K):
        for zs in range(K):
            num[zs] += px[xc] * Qs[xc, zs] * Qts[zs, int(z_t)]
    tot = num.sum()
    return None if tot == 0.0 else num / tot


def sequence_posterior_bruteforce(prior, xs, zt_seq, alpha_t, alpha_s):
    """Joint posterior over whole sequences z_s^{1:L} (dict: tuple -> prob).

    x_theta is a product over positions (one distribution per position) and
    the forward process acts independently on each position; the joint is
    enumerated without using that factorisation.
    """
    xs = [np.asarray(x, dtype=np.float64) for x in xs]
    V = xs[0].shape[0]
    pi = prior_vector(prior, V)
    K = pi.shape[0]
    Qs = transition(alpha_s, pi)
    Qts = transition(alpha_t / alpha_s, pi)
    L = len(xs)
    post = {}
    for zs in itertools.product(range(K), repeat=L):
        tot = 0.0
        for xseq in itertools.product(range(V), repeat=L):
            w = 1.0
            for l in range(L):
                w *= xs[l][xseq[l]] * Qs[xseq[l], zs[l]] * Qts[zs[l], int(zt_seq[l])]
            tot += w
        post[zs] = tot
    Z = sum(post.values())
    return {k: v / Z for k, v in post.items()}
