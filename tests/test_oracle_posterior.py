"""Pins of the oracle's reverse posteriors against Bayes' rule and the Psi forms."""
import itertools

import numpy as np
import pytest

from oracle import bayes, posterior, schedule

TS_PAIRS = [(1.0, 0.0), (1.0, 0.5), (0.75, 0.5), (0.5, 0.25), (0.3, 0.01),
            (1.0 / 128, 0.0), (0.9, 0.89)]


def _x(V, seed, peaked=False):
    r = np.random.default_rng(seed)
    a = 0.3 if peaked else 2.0
    return r.dirichlet(np.full(V, a))


def _alphas(t, s):
    return float(schedule.alpha(t)), float(schedule.alpha(s))


def check_against_bayes(post_fn, prior, V, seeds=(0, 1, 2)):
    """max |closed form - brute force| over all z_t, (t, s) pairs and seeds."""
    worst, compared = 0.0, 0
    K = V + 1 if prior == "mask" else V
    for seed in seeds:
        x = _x(V, seed, peaked=seed % 2 == 1)
        for t, s in TS_PAIRS:
            at, as_ = _alphas(t, s)
            for zt in range(K):
                bf = bayes.posterior_bruteforce(prior, x, zt, at, as_)
                if bf is None:          # z_t impossible at this t: nothing to compare
                    assert prior == "mask" and zt != V and at == 0.0
                    continue
                cf = post_fn(x, zt, at, as_)
                d = np.abs(bf - cf)
                assert np.all(np.isfinite(d))
                worst = max(worst, float(d.max()))
                compared += 1
    assert compared >= len(seeds) * (len(TS_PAIRS) - 2) * K
    return worst


@pytest.mark.parametrize("V", [2, 3, 5, 8])
def test_mdm_closed_form_equals_bayes(V):
    assert check_against_bayes(posterior.mdm_posterior, "mask", V) < 1e-12


@pytest.mark.parametrize("V", [2, 3, 5, 8])
def test_usdm_closed_form_equals_bayes(V):
    assert check_against_bayes(posterior.usdm_posterior, "uniform", V) < 1e-12


def test_forward_composition_defines_alpha_t_given_s():
    for prior, V in (("mask", 4), ("uniform", 5)):
        pi = bayes.prior_vector(prior, V)
        for t, s in TS_PAIRS:
            at, as_ = _alphas(t, s)
            if as_ == 0:
                continue
            lhs = bayes.transition(as_, pi) @ bayes.transition(schedule.alpha_t_given_s(at, as_), pi)
            assert np.allclose(lhs, bayes.transition(at, pi), atol=1e-14)


@pytest.mark.parametrize("prior,V", [("mask", 3), ("uniform", 3), ("uniform", 2)])
def test_sequence_posterior_factorises(prior, V):
    """Joint enumeration over whole sequences equals the product of per-position closed forms."""
    L = 2
    xs = [_x(V, 10 + l) for l in range(L)]
    K = V + 1 if prior == "mask" else V
    at, as_ = _alphas(0.6, 0.2)
    for zt in itertools.product(range(K), repeat=L):
        joint = bayes.sequence_posterior_bruteforce(prior, xs, zt, at, as_)
        per = [posterior.posterior(prior, xs[l], zt[l], at, as_) for l in range(L)]
        for zs, p in joint.items():
            assert abs(p - per[0][zs[0]] * per[1][zs[1]]) < 1e-12


@pytest.mark.parametrize("prior", ["mask", "uniform"])
def test_normalised_and_nonnegative(prior):
    V = 7
    K = V + 1 if prior == "mask" else V
    for seed in range(4):
        x = _x(V, seed)
        for t, s in TS_PAIRS:
            at, as_ = _alphas(t, s)
            for zt in range(K):
                p = posterior.posterior(prior, x, zt, at, as_)
                assert abs(p.sum() - 1.0) < 1e-12 and p.min() >= 0


def test_mdm_carry_over_and_alpha_s_one():
    V = 6
    x = _x(V, 3)
    for t in (1.0, 0.5, 0.1):
        at = float(schedule.alpha(t))
        for zt in range(V):
            p = posterior.mdm_posterior(x, zt, at, 0.7 if at < 0.7 else 1.0)
            assert p[zt] == 1.0 and p.sum() == 1.0
        p = posterior.mdm_posterior(x, V, at, 1.0)      # last step: no mask mass left
        assert p[V] == 0.0 and np.allclose(p[:V], x, atol=1e-15)


def test_usdm_alpha_s_one_reduction_and_positivity():
    V = 6
    x = _x(V, 4)
    for at in (0.0, 0.3, 0.9):
        for r in range(V):
            p = posterior.usdm_posterior(x, r, at, 1.0)
            w = np.full(V, 1.0 - at)
            w[r] += V * at
            assert np.allclose(p, x * w / (V * at * x[r] + 1.0 - at), atol=1e-14)
            q = posterior.usdm_posterior(x, r, at * 0.5, 0.95)   # alpha_s < 1: all classes reachable
            assert q.min() > 0


@pytest.mark.parametrize("prior", ["mask", "uniform"])
def test_single_step_s0_t1_is_x_theta(prior):
    """App. A.4 single-step reductions: s = 0, t = 1 gives Cat(x_theta)."""
    V = 9
    x = _x(V, 5)
    at, as_ = float(schedule.alpha(1.0)), float(schedule.alpha(0.0))
    if prior == "mask":
        p = posterior.mdm_posterior(x, V, at, as_)
        assert np.allclose(p[:V], x, atol=1e-15) and p[V] == 0
        for kappa in (0.0, 0.4, 1.0):
            for zt in (0, V):
                q = posterior.psi_mdm(x, zt, at, as_, kappa)
                assert np.allclose(q[:V], x, atol=1e-15) and abs(q[V]) < 1e-15
    else:
        for r in range(V):
            assert np.allclose(posterior.usdm_posterior(x, r, at, as_), x, atol=1e-15)
            for kappa in (0.0, 0.4, 1.0):
                assert np.allclose(posterior.psi_usdm(x, r, at, as_, kappa), x, atol=1e-15)


def test_psi_mdm_kappa_one_masked_equals_posterior():
    V = 5
    x = _x(V, 6)
    for t, s in TS_PAIRS:
        at, as_ = _alphas(t, s)
        assert np.allclose(posterior.psi_mdm(x, V, at, as_, 1.0),
                           posterior.mdm_posterior(x, V, at, as_), atol=1e-14)


@pytest.mark.parametrize("kappa", [0.0, 0.3, 0.8, 1.0])
def test_psi_closed_forms_equal_generic_mixture(kappa):
    """eq. (psi-mdm) / (psi-usdm) equal eq. (psi-sampler) built from the posteriors."""
    V = 5
    x = _x(V, 7)
    for t, s in TS_PAIRS:
        at, as_ = _alphas(t, s)
        pm = bayes.prior_vector("mask", V)
        for zt in range(V + 1):
            gen = posterior.psi_generic(posterior.mdm_posterior_plugin(x, zt, at, as_),
                                        posterior.mdm_posterior_plugin(x, zt, at, 1.0), pm, as_, kappa)
            assert np.allclose(posterior.psi_mdm(x, zt, at, as_, kappa), gen, atol=1e-14)
        pu = bayes.prior_vector("uniform", V)
        for r in range(V):
            gen = posterior.psi_generic(posterior.usdm_posterior(x, r, at, as_),
                                        posterior.usdm_posterior(x, r, at, 1.0), pu, as_, kappa)
            assert np.allclose(posterior.psi_usdm(x, r, at, as_, kappa), gen, atol=1e-14)
            if kappa == 1.0:
                assert np.allclose(posterior.psi_usdm(x, r, at, as_, 1.0),
                                   posterior.usdm_posterior(x, r, at, as_), atol=1e-14)


def test_schedule_endpoints():
    a = schedule.alphas(128)
    assert a[0] == 1.0 and a[-1] == 0.0 and np.all(np.diff(a) < 0)
