"""The T-step ancestral sampling loop (test infrastructure only).

App. A.1/A.2: generation applies the learned reverse posterior
p_theta(z_s | z_t) = q_{s|t}(z_s | z_t, x = x_theta(z_t, t)) repeatedly from
z_1 ~ prior to z_0.  With the grid t_k = k / T (schedule.py), step k = T .. 1
runs the denoiser at alpha_t = alphas[k] and samples z_{t_{k-1}} with
(alpha_t, alpha_s) = (alphas[k], alphas[k-1]); its noise is keyed by step k
(or, with explicit noise, read from noise_words[k - 1]).  This is App. A.4,
eq. (psi-sampler) at kappa_t = 1 (ancestral sampling); with kappas given, step k
applies the Psi transition with kappa_t = kappas[k] (sampler.psi_sample).

Pinned through its parts and by the bookkeeping invariants of the masked
prior: unmasked tokens never change, the masked count never increases, and no
mask remains after the last step (alpha_s = alpha_0 = 1).
"""
import numpy as np

from . import forward as _fw
from . import sampler as _sm


def sample_loop(cfg, P, z1, T, alphas, noise_seed=None, noise_words=None, kappas=None):
    """Returns (z_0 [B, L], trace [T + 1, B, L] with trace[0] = z_1, gaps [T, B*L, 2])."""
    z = np.array(z1, dtype=np.int64)
    B, L = z.shape
    prior, V = cfg["prior"], cfg["vocab"]
    trace = [z.copy()]
    gaps = []
    ntop = _sm.n_top(prior, V)
    for k in range(T, 0, -1):
        logits = _fw.forward(cfg, P, z, alphas[k]).reshape(B * L, V)
        if noise_words is not None:
            nz = _sm.ExplicitNoise(noise_words[k - 1], ntop)
        else:
            nz = _sm.PhiloxNoise(noise_seed, k)
        if kappas is None:
            zs, g = _sm.posterior_sample(prior, logits, z.reshape(-1), alphas[k], alphas[k - 1], nz)
        else:
            zs, g = _sm.psi_sample(prior, logits, z.reshape(-1), alphas[k], alphas[k - 1], kappas[k], nz)
        z = zs.reshape(B, L)
        trace.append(z.copy())
        gaps.append(g)
    return z, np.stack(trace), np.stack(gaps)
