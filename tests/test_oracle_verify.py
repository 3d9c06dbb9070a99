"""Pins of the speculative-verification oracle (Alg. 1, linear sampler)."""
import numpy as np
import pytest
from scipy import stats

from oracle import philox, sampler, verify


def _chi2(counts, probs):
    exp = probs * counts.sum()
    big = exp >= 5
    obs = list(counts[big]) + ([counts[~big].sum()] if (~big).any() else [])
    ex = list(exp[big]) + ([exp[~big].sum()] if (~big).any() else [])
    obs, ex = np.array(obs, float), np.array(ex, float)
    keep = ex > 0
    return stats.chisquare(obs[keep], ex[keep] * obs[keep].sum() / ex[keep].sum()).pvalue


def _logits(seed, shape, scale=1.5):
    return scale * np.random.default_rng(seed).standard_normal(shape)


def test_first_emitted_token_is_distributed_as_the_target():
    """Speculative sampling is lossless: with the draft token x_1 ~ q_1, the first emitted token
    (x_1 if accepted, else the residual draw) follows p_1 whatever q_1 is."""
    V, B, n = 12, 3, 30000
    pl = _logits(1, (B, V))
    ql = _logits(2, (B - 1, V)) + np.linspace(0, 2, V)      # a deliberately different proposal
    p1 = np.exp(pl[0] - pl[0].max()); p1 /= p1.sum()
    q1 = np.exp(ql[0] - ql[0].max()); q1 /= q1.sum()
    r = np.random.default_rng(3)
    first = np.empty(n, dtype=np.int64)
    for k in range(n):
        draft = np.array([r.choice(V, p=q1), r.choice(V, p=q1)])
        nn, z, _, _ = verify.verify_one(pl, ql, draft, k, verify.PhiloxVerifyNoise(9, 4))
        first[k] = draft[0] if nn > 1 else z
    assert _chi2(np.bincount(first, minlength=V), p1) > 1e-3


def test_identical_draft_and_target_accept_everything():
    V, B = 50, 6
    pl = _logits(4, (B, V))
    draft = np.arange(B - 1) * 3
    n, z, marg, _ = verify.verify_one(pl, pl[:-1], draft, 0, verify.PhiloxVerifyNoise(1, 1))
    assert n == B and np.all(marg <= 0)
    # the bonus token is then the plain two-level draw from p_B
    zb, _, _ = sampler.sample_from_probs("uniform", np.exp(pl[-1] - pl[-1].max()) / np.exp(pl[-1] - pl[-1].max()).sum(),
                                         0, verify.PhiloxVerifyNoise(1, 1))
    assert z == zb


def test_tpf_bounds_and_acceptance_rate():
    """1 <= TPF = (n + 1) / 2 <= (B + 1) / 2, and the acceptance probability of one position is
    sum_x min(p(x), q(x)) (1 - total variation distance)."""
    V, B, S = 20, 5, 6000
    pl = _logits(5, (S, B, V), scale=1.0)
    ql = pl[:, :-1] + _logits(6, (S, B - 1, V), scale=0.7)
    r = np.random.default_rng(7)
    q = np.exp(ql - ql.max(-1, keepdims=True)); q /= q.sum(-1, keepdims=True)
    draft = np.array([[r.choice(V, p=q[s, i]) for i in range(B - 1)] for s in range(S)])
    n, z, marg, _ = verify.spec_verify(pl, ql, draft, verify.PhiloxVerifyNoise(2, 8))
    tpf = (n + 1) / 2
    assert tpf.min() >= 1 and tpf.max() <= (B + 1) / 2
    p = np.exp(pl - pl.max(-1, keepdims=True)); p /= p.sum(-1, keepdims=True)
    acc = np.minimum(p[:, 0], q[:, 0]).sum(-1)                # per-sequence acceptance prob. of position 1
    first_ok = (n > 1).astype(float)
    # binomial z-test of the observed first-position acceptances against their expectation
    zscore = (first_ok.sum() - acc.sum()) / np.sqrt((acc * (1 - acc)).sum())
    assert abs(zscore) < 4


def test_explicit_noise_equals_philox_noise():
    V, B, S = 300, 4, 10
    pl, ql = _logits(8, (S, B, V)), _logits(9, (S, B - 1, V))
    draft = np.random.default_rng(1).integers(0, V, (S, B - 1))
    seqs = np.arange(S)[:, None]
    ntop = sampler.n_top("uniform", V)
    words = np.concatenate([philox.counter_words(11, philox.STREAM_VERIFY, 3, seqs, np.arange(B - 1)[None]),
                            philox.counter_words(11, philox.STREAM_TOP, 3, seqs, np.arange(ntop)[None]),
                            philox.counter_words(11, philox.STREAM_CLASS, 3, seqs, np.arange(V)[None])], 1)
    assert words.shape[1] == verify.noise_width(B, V)
    a = verify.spec_verify(pl, ql, draft, verify.PhiloxVerifyNoise(11, 3))
    b = verify.spec_verify(pl, ql, draft, verify.ExplicitVerifyNoise(words, B, V))
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_residual_excludes_classes_where_the_draft_is_likelier():
    """After a rejection the replacement never takes a class with q_n >= p_n."""
    V, B, S = 16, 2, 3000
    pl = _logits(12, (S, B, V))
    ql = _logits(13, (S, B - 1, V), scale=3.0)
    p = np.exp(pl[:, 0] - pl[:, 0].max(-1, keepdims=True)); p /= p.sum(-1, keepdims=True)
    q = np.exp(ql[:, 0] - ql[:, 0].max(-1, keepdims=True)); q /= q.sum(-1, keepdims=True)
    draft = np.argmax(q, -1)[:, None]                          # the draft's favourite: often rejected
    n, z, _, _ = verify.spec_verify(pl, ql, draft, verify.PhiloxVerifyNoise(5, 5))
    rej = n == 1
    assert rej.sum() > 100
    assert np.all(p[rej, z[rej]] > q[rej, z[rej]])
