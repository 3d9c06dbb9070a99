"""Planted mistakes in the oracle must be caught by its pins (CPU only).

Each test swaps one oracle function for a plausible wrong version (a sign, a
dropped term, an inverted ratio, a missing scale, a wrong transform) and
asserts that the corresponding pin rejects it.
"""
import numpy as np
import pytest

from oracle import forward, forward_loops, noise, philox, posterior, sampler
from tests.test_oracle_posterior import check_against_bayes
from tests.test_oracle_forward import CFG, _P, _z
from tests.test_oracle_sampler import chi2_pvalue, _peaked_probs


def _mdm_sign(x, z_t, at, as_):
    p = posterior.mdm_posterior(x, z_t, at, as_)
    if int(z_t) == x.shape[0]:
        p[:-1] = (at - as_) / (1 - at) * x
    return p


def _usdm_drop_uniform_term(x, z_t, at, as_):
    K = x.shape[0]
    a_ts = at / as_
    z = np.zeros(K)
    z[int(z_t)] = 1
    num = K * at * z * x + (a_ts - at) * z + (as_ - at) * x
    return num / (K * at * x[int(z_t)] + 1 - at)


def _usdm_inverted_ratio(x, z_t, at, as_):
    return posterior.usdm_posterior(x, z_t, at, as_) if as_ == 0 else \
        _usdm_with_ats(x, z_t, at, as_, as_ / max(at, 1e-300))


def _usdm_with_ats(x, z_t, at, as_, a_ts):
    K = x.shape[0]
    z = np.zeros(K)
    z[int(z_t)] = 1
    num = (K * at * z * x + (a_ts - at) * z + (as_ - at) * x + (1 - a_ts) * (1 - as_) / K)
    return num / (K * at * x[int(z_t)] + 1 - at)


@pytest.mark.parametrize("bad,prior", [(_mdm_sign, "mask"), (_usdm_drop_uniform_term, "uniform"),
                                       (_usdm_inverted_ratio, "uniform")])
def test_bayes_pin_catches_posterior_mistakes(bad, prior):
    with np.errstate(all="ignore"):
        try:
            worst = check_against_bayes(bad, prior, 4)
        except AssertionError:
            return                   # non-finite or inconsistent output: caught
    assert worst > 1e-6


def _forward_mismatch():
    P = _P(scale=20.0)
    z = _z()
    a = forward.forward(CFG, P, z, 0.37)
    b = np.array(forward_loops.forward_loops(CFG, P, z, 0.37))
    return np.abs(a - b).max()


def test_loop_pin_catches_missing_attention_scale(monkeypatch):
    def att(q, k, v, vis=None):
        s = q @ k.T
        p = np.exp(s - s.max(-1, keepdims=True))
        return (p / p.sum(-1, keepdims=True)) @ v
    monkeypatch.setattr(forward, "attention", att)
    assert _forward_mismatch() > 1e-6


def test_loop_pin_catches_wrong_gelu(monkeypatch):
    monkeypatch.setattr(forward, "gelu_tanh", lambda x: 0.5 * x * (1 + np.tanh(0.8 * (x + 0.044715 * x ** 3))))
    assert _forward_mismatch() > 1e-6


def test_loop_pin_catches_swapped_time_embedding(monkeypatch):
    orig = forward.time_embedding
    monkeypatch.setattr(forward, "time_embedding", lambda a, d: orig(a, d)[::-1].copy())
    assert _forward_mismatch() > 1e-6


def test_loop_pin_catches_centred_rms_norm(monkeypatch):
    """RMSNorm that removes the mean first (i.e. a shift-free LayerNorm) is caught by the scalar
    loops under norm = "rms"."""
    def rms(x, g, eps):
        c = x - x.mean(-1, keepdims=True)
        return c / np.sqrt((c ** 2).mean(-1, keepdims=True) + eps) * g
    monkeypatch.setattr(forward, "rms_norm", rms)
    cfg = dict(CFG, norm="rms")
    P = _P(cfg, scale=20.0)
    z = _z()
    a = forward.forward(cfg, P, z, 0.37)
    b = np.array(forward_loops.forward_loops(cfg, P, z, 0.37))
    assert np.abs(a - b).max() > 1e-6


def test_loop_pin_catches_unbiased_variance(monkeypatch):
    def ln(x, g, b, eps):
        mu = x.mean(-1, keepdims=True)
        return (x - mu) / np.sqrt(x.var(-1, ddof=1, keepdims=True) + eps) * g + b
    monkeypatch.setattr(forward, "layer_norm", ln)
    assert _forward_mismatch() > 1e-6


def test_chi2_pin_catches_gumbel_sign(monkeypatch):
    monkeypatch.setattr(noise, "gumbel", lambda w: np.log(noise.exponential(w)))
    V = 40
    p = _peaked_probs("uniform", V, 2)
    n = 20000
    w = philox.counter_words(5, 9, 0, np.arange(n)[:, None], np.arange(V)[None, :])
    z = np.array([sampler.sample_flat(p, w[i]) for i in range(n)])
    assert chi2_pvalue(np.bincount(z, minlength=V), p) < 1e-6


def test_kat_pin_catches_wrong_multiplier(monkeypatch):
    monkeypatch.setattr(philox, "_M0", 0xD2511F55)
    assert philox.philox_scalar((0, 0, 0, 0), (0, 0))[0] != 0x6627e8d5


def test_lossless_pin_catches_a_wrong_residual(monkeypatch):
    """Replacing the residual [p - q]_+ by [q - p]_+, or by p itself, must break the lossless
    chi-square pin of the speculative verification."""
    from oracle import verify
    from tests import test_oracle_verify as tv

    def make_wrong(kind):
        def wrong_verify_one(p_logits, q_logits, draft, seq, nz):
            B, V = p_logits.shape
            u = verify.word_uniform(nz.accept(seq, B - 1))
            n = B
            for i in range(B - 1):
                p, q = verify._softmax(p_logits[i]), verify._softmax(q_logits[i])
                if u[i] > min(1.0, p[draft[i]] / q[draft[i]]):
                    n = i + 1
                    break
            if n == B:
                dist = verify._softmax(p_logits[B - 1])
            else:
                p, q = verify._softmax(p_logits[n - 1]), verify._softmax(q_logits[n - 1])
                dist = np.maximum(q - p, 0.0) if kind == "swapped" else p
                dist = dist / dist.sum()
            z, g1, g2 = sampler.sample_from_probs("uniform", dist, seq, nz)
            return n, z, None, (g1, g2)
        return wrong_verify_one

    for kind in ("swapped", "plain_p"):
        monkeypatch.setattr(verify, "verify_one", make_wrong(kind))
        with pytest.raises(AssertionError):
            tv.test_first_emitted_token_is_distributed_as_the_target()


def test_pattern_pins_catch_transposed_visibility(monkeypatch):
    """A pattern applied as vis^T (keys and queries swapped) fails the scalar-loop pin."""
    from tests import test_oracle_masked_lora as t
    orig = forward.attention
    monkeypatch.setattr(forward, "attention", lambda q, k, v, vis=None: orig(q, k, v, None if vis is None else vis.T))
    with pytest.raises(AssertionError):
        t.test_masked_forward_equals_scalar_loops("causal")


def test_lora_pins_catch_wrong_adapter_scale(monkeypatch):
    """r / alpha in place of alpha / r fails the merged-weight identity."""
    from tests import test_oracle_masked_lora as t
    orig = forward.projection

    def proj(cfg, P, l, name, a, gate):
        if cfg.get("lora_rank"):
            cfg = dict(cfg, lora_alpha=cfg["lora_rank"] ** 2 / cfg["lora_alpha"])
        return orig(cfg, P, l, name, a, gate)
    monkeypatch.setattr(forward, "projection", proj)
    with pytest.raises(AssertionError):
        t.test_all_gates_on_equals_merged_weights()


def test_lora_pins_catch_gate_on_the_wrong_positions(monkeypatch):
    """A gate indexed from the end of the sequence fails the teacher property of the [x, z_1] pass."""
    from tests import test_oracle_masked_lora as t
    orig = forward.projection
    monkeypatch.setattr(forward, "projection", lambda cfg, P, l, name, a, gate: orig(cfg, P, l, name, a, gate[::-1]))
    with pytest.raises(AssertionError):
        t.test_teacher_logits_from_one_pass_over_x_and_z()


def test_exact_pin_catches_reversed_inverse_cdf(monkeypatch):
    """An inverse CDF that scans the group from its last class has the same distribution (chi-square
    cannot see it) but a different map from the uniform to the class: the exact-rational pin fails."""
    from tests.test_oracle_sampler import check_inverse_cdf_against_exact
    orig = sampler.inverse_cdf

    def reversed_cdf(w, word):
        w = np.asarray(w, dtype=np.float64)
        j, gap = orig(w[::-1], word)
        return len(w) - 1 - j, gap
    monkeypatch.setattr(sampler, "inverse_cdf", reversed_cdf)
    assert check_inverse_cdf_against_exact(n=500) > 50

