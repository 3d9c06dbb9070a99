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


def test_mask_first_reads_the_mask_word_and_compares_below():
    """Stage 0 of the masked draw: the mask is taken iff the uniform of level-1 word n_groups is
    below p_V (words chosen just below and just above the threshold; every other word fixed).
    Pins the word index, the direction of the comparison and that the other words are not read."""
    V = 600
    ng = sampler.n_groups_real(V)
    p = np.zeros(V + 1)
    p[:V] = 0.7 / V
    p[V] = 0.3
    thr = int(0.3 * 2.0 ** 32)                # u(w) = (w + 1/2) 2^-32
    for w, expect_mask in ((thr - 1, True), (thr + 1, False)):
        for other in (0, 2 ** 32 - 1):
            words = np.full((1, sampler.noise_width("mask", V)), other, dtype=np.uint32)
            words[0, ng] = w
            nz = sampler.ExplicitNoise(words, sampler.n_top("mask", V))
            # (level 2' reads Philox uniforms, which explicit words do not carry: the inverse-CDF
            # draw is checked where stage 0 ends it)
            draws = (sampler.sample_from_probs,) + ((sampler.sample_from_probs_cdf,) if expect_mask else ())
            for draw in draws:
                z, g0, _ = draw("mask", p, 0, nz)
                assert (z == V) == expect_mask, (draw.__name__, w, other, z)
                assert g0 < 1e-8          # the reported gap covers the near-tie with p_V


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


# ---------------------------------------------------------------- level 2' (inverse CDF in the group)

def inverse_cdf_exact(w, word):
    """The class u * sum(w) falls in, in exact rational arithmetic (u = (word + 1/2) 2^-32): the
    first j with w_0 + .. + w_j > u * sum(w).  Integer weights only."""
    from fractions import Fraction
    S = sum(int(x) for x in w)
    t = Fraction(2 * int(word) + 1, 2 ** 33) * S
    c = 0
    for j, x in enumerate(w):
        c += int(x)
        if c > t:
            return j
    raise AssertionError("u < 1 always falls inside")


def check_inverse_cdf_against_exact(n=3000, seed=7):
    """Number of random integer-weight groups (with zero weights mixed in) on which
    sampler.inverse_cdf disagrees with the exact rational answer (away from boundaries)."""
    r = np.random.default_rng(seed)
    bad = 0
    for _ in range(n):
        k = int(r.integers(1, 12))
        w = r.integers(0, 6, size=k)
        if w.sum() == 0:
            w[int(r.integers(0, k))] = 1
        word = int(r.integers(0, 2 ** 32))
        j, gap = sampler.inverse_cdf(w.astype(float), word)
        if gap > 1e-12 and j != inverse_cdf_exact(w, word):
            bad += 1
    return bad


def test_inverse_cdf_equals_exact_rational_answer():
    assert check_inverse_cdf_against_exact() == 0
    # fixed cases: u just below 1/2 and just above, on weights (1, 1, 2); a zero weight is skipped
    assert sampler.inverse_cdf([1.0, 1.0, 2.0], 2 ** 31 - 1)[0] == 1
    assert sampler.inverse_cdf([1.0, 1.0, 2.0], 2 ** 31)[0] == 2
    assert sampler.inverse_cdf([0.0, 3.0, 0.0, 1.0], 0)[0] == 1
    assert sampler.inverse_cdf([0.0, 3.0, 0.0, 1.0], 2 ** 32 - 1)[0] == 3


def draw_many_cdf(prior, p, n, seed=13):
    out = np.empty(n, dtype=np.int64)
    for i in range(n):
        out[i] = sampler.sample_from_probs_cdf(prior, p, 3, sampler.PhiloxNoise(seed, i))[0]
    return out


@pytest.mark.parametrize("prior", ["mask", "uniform"])
def test_inverse_cdf_draws_match_posterior_chi2(prior):
    V = 600                                    # three real groups (256, 256, 88)
    p = _peaked_probs(prior, V, 3)
    z = draw_many_cdf(prior, p, 20000)
    counts = np.bincount(z, minlength=p.shape[0])
    assert chi2_pvalue(counts, p) > 1e-3
    gb = sampler.group_bounds(prior, V)
    gc = np.array([counts[a:b].sum() for a, b in gb])
    gp = np.array([p[a:b].sum() for a, b in gb])
    assert chi2_pvalue(gc, gp) > 1e-3


def test_inverse_cdf_and_gumbel_draws_pick_the_same_group():
    """Level 1 is shared: on the same noise both readings choose the same group every time."""
    V = 700
    p = _peaked_probs("mask", V, 4)
    bounds = sampler.group_bounds("mask", V)
    grp = lambda z: next(i for i, (a, b) in enumerate(bounds) if a <= z < b)
    for i in range(400):
        nz = sampler.PhiloxNoise(21, i)
        a = sampler.sample_from_probs("mask", p, 5, nz)[0]
        b = sampler.sample_from_probs_cdf("mask", p, 5, nz)[0]
        assert grp(a) == grp(b)


def test_group_candidates_follow_the_group_softmax_chi2():
    """Each group's candidate, over many rows (independent uniforms), is distributed as the
    softmax of the group's logits; the last group is ragged."""
    V = 300
    l = 2.0 * np.random.default_rng(8).standard_normal(V)
    n = 12000
    cands = np.array([sampler.group_candidates(l, row, sampler.PhiloxNoise(17, 2), V)[0] for row in range(n)])
    for g, (a, b) in enumerate(sampler.group_bounds("uniform", V)):
        w = np.exp(l[a:b] - l[a:b].max())
        counts = np.bincount(cands[:, g] - a, minlength=b - a)
        assert chi2_pvalue(counts, w / w.sum()) > 1e-3


def test_posterior_sample_cdf_masked_rows_and_carry_over():
    """posterior_sample with level 2': unmasked rows carried over, masked rows drawn inside the
    group level 1 picks, the draw equal to sample_from_probs_cdf on the row's posterior."""
    V, R = 520, 40
    r = np.random.default_rng(9)
    logits = r.standard_normal((R, V)) * 2
    z_t = np.where(r.random(R) < 0.6, V, r.integers(0, V, R))
    nz = sampler.PhiloxNoise(33, 4)
    zs, gaps = sampler.posterior_sample("mask", logits, z_t, 0.3, 0.6, nz, level2="cdf")
    for i in range(R):
        if z_t[i] != V:
            assert zs[i] == z_t[i]
            continue
        x = np.exp(logits[i] - logits[i].max())
        p = posterior.posterior("mask", x / x.sum(), V, 0.3, 0.6)
        assert zs[i] == sampler.sample_from_probs_cdf("mask", p, i, nz)[0]
    with pytest.raises(ValueError):
        sampler.posterior_sample("mask", logits, z_t, 0.3, 0.6, nz, level2="flat")
