"""Reverse posteriors p_{s|t}(z_s | z_t, x_theta) in float64 (test infrastructure only).

Notation: V real tokens; for the masked prior the mask is class V (the K-th
category, Background: Notation), so K = V + 1 classes; for the uniform prior
K = V.  `x` is a probability vector over the V real tokens (x_theta of one
position), z_t an integer class id.

mdm_posterior      App. A.1, eq. (mdm-posterior), with the learned plug-in
                   x = x_theta.  Masked z_t: (a_s - a_t)/(1 - a_t) x +
                   (1 - a_s)/(1 - a_t) m.  Unmasked z_t: carry-over, z_s = z_t
                   (App. A.1: unmasked tokens stay unchanged and this carries
                   over to the reverse process; they cannot be remasked).
mdm_posterior_plugin   the same equation read literally for unmasked z_t,
                   Cat(x_theta); used only to check the Psi closed form.
usdm_posterior     App. A.2, eq. (uniform_true_reverse_posterior) with x = x_theta.
psi_generic        App. A.4, eq. (psi-sampler): kappa q_{s|t} + (1 - kappa)
                   [a_s q_{0|t} + (1 - a_s) pi].
psi_mdm, psi_usdm  App. A.4, eqs. (psi-mdm) and (psi-usdm), typed from their
                   printed closed forms.

Pinned by brute-force Bayes enumeration of the forward process (bayes.py),
by kappa = 1 agreement of the Psi forms, by normalisation, and by the s = 0,
t = 1 single-step reductions (eqs. (psi-mdm-single-step), (psi-usdm-single-step)).
"""
import numpy as np


def mdm_posterior(x, z_t, alpha_t, alpha_s):
    """Probabilities over V + 1 classes (mask = index V) for one position."""
    x = np.asarray(x, dtype=np.float64)
    V = x.shape[-1]
    p = np.zeros(V + 1)
    if int(z_t) == V:
        p[:V] = (alpha_s - alpha_t) / (1.0 - alpha_t) * x
        p[V] = (1.0 - alpha_s) / (1.0 - alpha_t)
    else:
        p[int(z_t)] = 1.0
    return p


def mdm_posterior_plugin(x, z_t, alpha_t, alpha_s):
    x = np.asarray(x, dtype=np.float64)
    V = x.shape[-1]
    if int(z_t) == V:
        return mdm_posterior(x, z_t, alpha_t, alpha_s)
    p = np.zeros(V + 1)
    p[:V] = x
    return p


def usdm_posterior(x, z_t, alpha_t, alpha_s):
    """Probabilities over K = V classes for one position with current state r = z_t."""
    x = np.asarray(x, dtype=np.float64)
    K = x.shape[-1]
    r = int(z_t)
    a_ts = alpha_t / alpha_s
    z = np.zeros(K)
    z[r] = 1.0
    num = (K * alpha_t * z * x + (a_ts - alpha_t) * z + (alpha_s - alpha_t) * x
           + (1.0 - a_ts) * (1.0 - alpha_s) / K)
    den = K * alpha_t * x[r] + 1.0 - alpha_t
    return num / den


def psi_generic(q_st, q_0t, prior, alpha_s, kappa):
    return kappa * q_st + (1.0 - kappa) * (alpha_s * q_0t + (1.0 - alpha_s) * prior)


def psi_mdm(x, z_t, alpha_t, alpha_s, kappa):
    x = np.asarray(x, dtype=np.float64)
    V = x.shape[-1]
    p = np.zeros(V + 1)
    if int(z_t) != V:
        p[:V] = (alpha_s + kappa * (1.0 - alpha_s)) * x
        p[V] = (1.0 - kappa) * (1.0 - alpha_s)
    else:
        c = kappa * alpha_t * (1.0 - alpha_s) / (1.0 - alpha_t)
        p[:V] = (alpha_s - c) * x
        p[V] = 1.0 - alpha_s + c
    return p


def psi_usdm(x, z_t, alpha_t, alpha_s, kappa):
    x = np.asarray(x, dtype=np.float64)
    K = x.shape[-1]
    r = int(z_t)
    a_ts = alpha_t / alpha_s
    z = np.zeros(K)
    z[r] = 1.0
    zx = x[r]
    den = K * alpha_t * zx + 1.0 - alpha_t
    num = (K * alpha_t * (alpha_s + kappa * (1.0 - alpha_s)) * z * x
           + kappa * (1.0 - alpha_s) * a_ts * z
           + (alpha_s * (1.0 - alpha_t) - kappa * alpha_t * (1.0 - alpha_s)) * x
           + (1.0 - alpha_s) * (kappa * (1.0 - a_ts) + (1.0 - kappa) * den) / K)
    return num / den


def posterior(prior, x, z_t, alpha_t, alpha_s):
    if prior == "mask":
        return mdm_posterior(x, z_t, alpha_t, alpha_s)
    if prior == "uniform":
        return usdm_posterior(x, z_t, alpha_t, alpha_s)
    raise ValueError(prior)
