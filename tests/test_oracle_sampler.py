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
    w = workloads.WORKLOADS[1]
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


# ---------------------------------------------------------------- Psi sampler (kappa < 1)

@pytest.mark.parametrize("prior", ["mask", "uniform"])
def test_psi_sample_at_kappa_one_is_the_ancestral_step(prior):
    V, R = 300, 24
    logits = workloads.synthetic_logits(21, R, V)
    if prior == "mask":
        zt = workloads.masked_state(22, 1, R, V, 0.6).reshape(-1)
    else:
        zt = workloads.uniform_state(22, 1, R, V).reshape(-1)
    a, _ = sampler.posterior_sample(prior, logits, zt, 0.3, 0.45, sampler.PhiloxNoise(4, 7))
    b, _ = sampler.psi_sample(prior, logits, zt, 0.3, 0.45, 1.0, sampler.PhiloxNoise(4, 7))
    assert np.array_equal(a, b)


def test_psi_unmasked_token_keep_or_remask_chi2():
    """Masked prior, unmasked z_t: eq. (psi-mdm) with x_theta = one-hot(z_t) keeps the token with
    probability a_s + kappa (1 - a_s) and remasks otherwise; the logits are never read."""
    V, n, at, as_, kappa = 40, 20000, 0.35, 0.5, 0.3
    logits = np.full((n, V), np.nan)                     # unread
    zt = np.full(n, 17)
    z, _ = sampler.psi_sample("mask", logits, zt, at, as_, kappa, sampler.PhiloxNoise(3, 2))
    assert set(np.unique(z)) <= {17, V}
    keep = as_ + kappa * (1 - as_)
    counts = np.array([(z == 17).sum(), (z == V).sum()])
    assert chi2_pvalue(counts, np.array([keep, 1 - keep])) > 1e-3


@pytest.mark.parametrize("prior", ["mask", "uniform"])
@pytest.mark.parametrize("kappa", [0.0, 0.45])
def test_psi_draws_match_psi_probabilities_chi2(prior, kappa):
    V, n = 600, 20000                                    # three real groups
    r = np.random.default_rng(5)
    l = 1.5 * r.standard_normal(V)
    l[r.integers(0, V, 3)] += 4.0
    x = np.exp(l - l.max())
    x /= x.sum()
    zt = V if prior == "mask" else 123
    f = posterior.psi_mdm if prior == "mask" else posterior.psi_usdm
    p = f(x, zt, 0.4, 0.55, kappa)
    z = np.empty(n, dtype=np.int64)
    for i in range(n):
        z[i] = sampler.sample_from_probs(prior, p, 3, sampler.PhiloxNoise(13, i))[0]
    assert chi2_pvalue(np.bincount(z, minlength=p.shape[0]), p) > 1e-3
    # the draw routine on a logit row gives exactly these probabilities
    _, _, pr = sampler.psi_sample(prior, l[None, :], np.array([zt]), 0.4, 0.55, kappa,
                                  sampler.PhiloxNoise(13, 0), return_probs=True)
    assert np.allclose(pr[0], p, rtol=0, atol=1e-15)


def test_psi_loop_bookkeeping_masked_config1():
    """kappa < 1 lets decoded tokens be remasked, tokens change only by unmasking or remasking, and
    the last step (a_s = 1) still leaves no mask."""
    c = 1
    cfg = workloads.model_cfg(c)
    V, T = cfg["vocab"], 8
    P = workloads.host_params(cfg, workloads.seeds(c)["param"], params.specs(cfg))
    z1 = workloads.all_mask(4, 32, V)
    al = schedule.alphas(T)
    kap = np.full(T + 1, 0.3)
    z0, trace, _ = loop.sample_loop(cfg, P, z1, T, al, noise_seed=9, kappas=kap)
    assert (trace[-1] == V).sum() == 0
    remasked = sum(int(((a != V) & (b == V)).sum()) for a, b in zip(trace[:-1], trace[1:]))
    assert remasked > 0                                   # decoded tokens were remasked
    for a, b in zip(trace[:-1], trace[1:]):
        changed = a != b
        # a change is either mask -> token or token -> mask
        assert np.all((a[changed] == V) ^ (b[changed] == V))
