"""Pins of the oracle's categorical sampler, Gaussian latent and loop bookkeeping."""
import math

import numpy as np
import pytest
from scipy import stats
from scipy.special import ndtr

from oracle import latent, loop, params, philox, posterior, sampler, schedule
import workloads


def chi2_pvalue(counts, probs):
    """Chi-square goodness of fit, merging classes with expected count < 5."""
    n = counts.sum()
    exp = probs * n
    big = exp >= 5
    obs_b, exp_b = list(counts[big]), list(exp[big])
    if (~big).any():
        obs_b.append(counts[~big].sum())
        exp_b.append(exp[~big].sum())
    obs_b, exp_b = np.array(obs_b, float), np.array(exp_b, float)
    # any class with zero probability must never be drawn
    assert counts[probs == 0].sum() == 0
    keep = exp_b > 0
    return stats.chisquare(obs_b[keep], exp_b[keep] * obs_b[keep].sum() / exp_b[keep].sum()).pvalue


def _peaked_probs(prior, V, seed):
    r = np.random.default_rng(seed)
    logits = 1.5 * r.standard_normal(V)
    logits[r.integers(0, V, 3)] += 4.0
    x = np.exp(logits - logits.max())
    x /= x.sum()
    at, as_ = 0.4, 0.55
    zt = V if prior == "mask" else int(r.integers(0, V))
    return posterior.posterior(prior, x, zt, at, as_)


def draw_many(prior, p, n, seed=11):
    out = np.empty(n, dtype=np.int64)
    for i in range(n):
        out[i] = sampler.sample_from_probs(prior, p, 3, sampler.PhiloxNoise(seed, i))[0]
    return out


@pytest.mark.parametrize("prior", ["mask", "uniform"])
def test_two_level_draws_match_posterior_chi2(prior):
    V = 600                                    # three real groups (256, 256, 88)
    p = _peaked_probs(prior, V, 1)
    z = draw_many(prior, p, 20000)
    counts = np.bincount(z, minlength=p.shape[0])
    assert chi2_pvalue(counts, p) > 1e-3
    # the level-1 (group) choice alone
    gb = sampler.group_bounds(prior, V)
    gc = np.array([counts[a:b].sum() for a, b in gb])
    gp = np.array([p[a:b].sum() for a, b in gb])
    assert chi2_pvalue(gc, gp) > 1e-3


def test_flat_gumbel_draws_match_chi2():
    V = 40
    p = _peaked_probs("uniform", V, 2)
    n = 20000
    w = philox.counter_words(5, 9, 0, np.arange(n)[:, None], np.arange(V)[None, :])
    z = np.array([sampler.sample_flat(p, w[i]) for i in range(n)])
    assert chi2_pvalue(np.bincount(z, minlength=V), p) > 1e-3


def test_explicit_noise_equals_philox_noise():
    V, R = 300, 12
    logits = workloads.synthetic_logits(3, R, V)
    zt = workloads.masked_state(4, 1, R, V, 0.7).reshape(-1)
    ntop = sampler.n_top("mask", V)
    rows = np.arange(R)
    words = np.concatenate([philox.counter_words(8, philox.STREAM_TOP, 5, rows[:, None], np.arange(ntop)[None]),
                            philox.counter_words(8, philox.STREAM_CLASS, 5, rows[:, None], np.arange(V)[None])], axis=1)
    a, _ = sampler.posterior_sample("mask", logits, zt, 0.3, 0.5, sampler.PhiloxNoise(8, 5))
    b, _ = sampler.posterior_sample("mask", logits, zt, 0.3, 0.5, sampler.ExplicitNoise(words, ntop))
    assert np.array_equal(a, b)
    assert words.shape[1] == sampler.noise_width("mask", V)


def test_carry_over_ignores_poisoned_rows():
    V, R = 50, 16
    logits = workloads.synthetic_logits(5, R, V)
    zt = workloads.masked_state(6, 1, R, V, 0.5).reshape(-1)
    keep = zt != V
    poisoned = logits.copy()
    poisoned[keep] = np.nan
    a, _ = sampler.posterior_sample("mask", logits, zt, 0.2, 0.6, sampler.PhiloxNoise(1, 3))
    b, _ = sampler.posterior_sample("mask", poisoned, zt, 0.2, 0.6, sampler.PhiloxNoise(1, 3))
    assert np.array_equal(a, b) and np.array_equal(a[keep], zt[keep])


def test_last_step_unmasks_everything():
    V, R = 70, 40
    logits = workloads.synthetic_logits(7, R, V)
    zt = workloads.masked_state(8, 1, R, V, 0.9).reshape(-1)
    z, _ = sampler.posterior_sample("mask", logits, zt, 1.0 / 64, 1.0, sampler.PhiloxNoise(2, 1))
    assert (z != V).all() and (z < V).all()


# --- Gaussian latent -------------------------------------------------------

def test_latent_k2_closed_form():
    """For K = 2, P(z = x) = P(eps' - eps < c) = Phi(c / sqrt 2), c = alpha_tilde / sigma."""
    for at in (0.0, 0.2, 0.5, 0.8):
        c = at / math.sqrt(1 - at * at)
        assert abs(latent.p_keep(at, 2) - ndtr(c / math.sqrt(2))) < 1e-10


def test_latent_alpha_map_endpoints_and_inverse():
    K = 50257
    assert abs(latent.alpha_of_tilde(0.0, K)) < 1e-9
    assert latent.alpha_of_tilde(0.999, K) > 0.999
    for a in (0.1, 0.5, 0.9):
        at = latent.tilde_of_alpha(a, K)
        assert abs(latent.alpha_of_tilde(at, K) - a) < 1e-8


def test_latent_uniform_at_zero_signal():
    V, R = 7, 6000
    x = np.zeros(R, dtype=np.int64)
    z = latent.latent_argmax(x, V, 0.0, 1.0, seed=3, step=0)
    assert chi2_pvalue(np.bincount(z, minlength=V), np.full(V, 1.0 / V)) > 1e-3


@pytest.mark.parametrize("at", [0.3, 0.6])
def test_latent_keep_probability_matches_quadrature(at):
    V, R = 8, 6000
    x = workloads.clean_tokens(9, 1, R, V).reshape(-1)
    z = latent.latent_argmax(x, V, at, math.sqrt(1 - at * at), seed=4, step=1)
    keep = (z == x)
    p = latent.p_keep(at, V)
    zscore = (keep.sum() - R * p) / math.sqrt(R * p * (1 - p))
    assert abs(zscore) < 4.0
    # non-kept outcomes are uniform over the other V - 1 classes
    off = (z[~keep] - x[~keep]) % V
    assert chi2_pvalue(np.bincount(off, minlength=V)[1:], np.full(V - 1, 1.0 / (V - 1))) > 1e-3


# --- loop bookkeeping -----------------------------------------------------

def _tiny_cfg():
    return workloads.model_cfg(1)


def test_loop_bookkeeping_masked_config1():
    cfg = _tiny_cfg()
    w = workloads.CONFIGS[1]
    P = params.init_params(cfg, workloads.seeds(1)["param"])
    B, L, V, T = w["B"], w["L"], w["vocab"], w["T"]
    words = workloads.noise_words(workloads.seeds(1)["noise"], (T, B * L, sampler.noise_width("mask", V)))
    z0, trace, _ = loop.sample_loop(cfg, P, workloads.all_mask(B, L, V), T, schedule.alphas(T), noise_words=words)
    assert (z0 != V).all() and (z0 >= 0).all()
    masked = (trace == V).sum(axis=(1, 2))
    assert np.all(np.diff(masked) <= 0) and masked[0] == B * L and masked[-1] == 0
    for k in range(1, T + 1):
        was = trace[k - 1] != V
        assert np.array_equal(trace[k][was], trace[k - 1][was])
    # deterministic
    z1, _, _ = loop.sample_loop(cfg, P, workloads.all_mask(B, L, V), T, schedule.alphas(T), noise_words=words)
    assert np.array_equal(z0, z1)


def test_loop_uniform_prior_runs():
    cfg = workloads.model_cfg(1, prior="uniform")
    P = params.init_params(cfg, 5)
    B, L, V, T = 2, 8, cfg["vocab"], 4
    z1 = workloads.uniform_state(3, B, L, V)
    z0, trace, _ = loop.sample_loop(cfg, P, z1, T, schedule.alphas(T), noise_seed=17)
    assert z0.shape == (B, L) and (trace >= 0).all() and (trace < V).all()
