"""Categorical sampling of z_s from the reverse posterior (test infrastructure only).

The paper draws each token of z_s from its per-position categorical
(App. A.4: the transition is applied token-wise; Sec. 4 linear sampler: each
position is drawn independently) but does not say how a categorical draw is
made.  The reading adopted here is a two-level Gumbel-max draw, exact for any
partition of the classes into groups:

  groups     real classes in contiguous groups of GROUP = 256
             ([0,256), [256,512), ..., [.., V)); for the masked prior the
             mask class V is one more, singleton group (the last one).
  level 1    g* = argmax_g  log M_g + G_g,   M_g = sum_{j in g} p_j,
             G_g = Gumbel of word (STREAM_TOP, step, row, g).
  level 2    z_s = argmax_{j in g*}  log p_j + G_j,
             G_j = Gumbel of word (STREAM_CLASS, step, row, j).
  ties       the lowest index wins at both levels; log 0 = -inf.

Exactness: the maximum over a group of log p_j + G_j is distributed as
log M_g plus a standard Gumbel and is independent of the group's argmax, so
level 1 picks group g with probability M_g and level 2 picks j with
probability p_j / M_g (the Gumbel-max property; Maddison, Tarlow, Minka,
"A* sampling", NeurIPS 2014, sec. 3).

Explicit-noise layout per row: NU = n_top + V words, the n_top level-1
words first, then one level-2 word per real class.

psi_sample draws from the Psi transition (App. A.4, eq. (psi-sampler), in the
closed forms eqs. (psi-mdm) and (psi-usdm)) with correction strength kappa in
[0, 1]; kappa = 1 is the ancestral step above.  For the masked prior an
unmasked position's x_theta is the one-hot of its token (the carry-over
parameterisation that makes kappa = 1 keep it), so under eq. (psi-mdm) the
token is kept with probability a_s + kappa (1 - a_s) and remasked with
probability (1 - kappa)(1 - a_s); its logits are never read.

Pinned by chi-square tests of many draws against the enumerated posterior and
against the flat (one Gumbel per class) Gumbel-max draw; psi_sample by equality
with posterior_sample at kappa = 1 and chi-square tests of its draws.
"""
import numpy as np

from . import noise as _nz
from . import philox as _ph
from . import posterior as _post

GROUP = 256


def n_groups_real(V):
    return (V + GROUP - 1) // GROUP


def n_top(prior, V):
    return n_groups_real(V) + (1 if prior == "mask" else 0)


def noise_width(prior, V):
    return n_top(prior, V) + V


def group_bounds(prior, V):
    b = [(g * GROUP, min((g + 1) * GROUP, V)) for g in range(n_groups_real(V))]
    if prior == "mask":
        b.append((V, V + 1))
    return b


class PhiloxNoise:
    """Noise words generated from (seed, step) with the counter layout of philox.py."""

    def __init__(self, seed, step):
        self.seed, self.step = int(seed), int(step)

    def top(self, row, count):
        return _ph.counter_words(self.seed, _ph.STREAM_TOP, self.step, row, np.arange(count))

    def cls(self, row, idx):
        return _ph.counter_words(self.seed, _ph.STREAM_CLASS, self.step, row, np.asarray(idx))


class ExplicitNoise:
    """Noise words read from a [rows, NU] uint32 array (level-1 words first)."""

    def __init__(self, words, ntop):
        self.words = np.asarray(words, dtype=np.uint32)
        self.ntop = ntop

    def top(self, row, count):
        return self.words[row, :count]

    def cls(self, row, idx):
        return self.words[row, self.ntop + np.asarray(idx)]


def _first_argmax_and_gap(scores):
    """Index of the first maximum and the gap to the runner-up (inf if none)."""
    i = int(np.argmax(scores))
    if scores.shape[0] < 2 or not np.isfinite(scores[i]):
        return i, np.inf
    rest = np.delete(scores, i)
    second = rest.max()
    return i, float(scores[i] - second) if np.isfinite(second) else np.inf


def sample_from_probs(prior, p, row, noise):
    """Two-level Gumbel-max draw from probabilities p over K classes.

    Returns (class id, level-1 gap, level-2 gap)."""
    V = p.shape[0] - (1 if prior == "mask" else 0)
    bounds = group_bounds(prior, V)
    with np.errstate(divide="ignore"):
        logM = np.log(np.array([p[a:b].sum() for a, b in bounds]))
        G = _nz.gumbel(noise.top(row, len(bounds)))
        g, gap1 = _first_argmax_and_gap(logM + G)
        a, b = bounds[g]
        if prior == "mask" and a == V:
            return V, gap1, np.inf
        idx = np.arange(a, b)
        s = np.log(p[a:b]) + _nz.gumbel(noise.cls(row, idx))
    j, gap2 = _first_argmax_and_gap(s)
    return a + j, gap1, gap2


def sample_flat(p, words):
    """Textbook one-Gumbel-per-class draw (used only to pin the two-level draw)."""
    with np.errstate(divide="ignore"):
        return int(np.argmax(np.log(p) + _nz.gumbel(words)))


def posterior_sample(prior, logits, z_t, alpha_t, alpha_s, noise, rows=None, return_probs=False):
    """One reverse step on a [R, V] logit matrix.

    Masked prior: rows whose z_t is not the mask id V are carried over.
    Returns z_s [R] (int64), the per-row level gaps [R, 2] and, optionally,
    the posterior probabilities [R, K].
    """
    logits = np.asarray(logits, dtype=np.float64)
    z_t = np.asarray(z_t)
    R, V = logits.shape
    rows = np.arange(R) if rows is None else np.asarray(rows)
    out = np.array(z_t, dtype=np.int64).copy()
    gaps = np.full((R, 2), np.inf)
    K = V + 1 if prior == "mask" else V
    probs = np.zeros((R, K)) if return_probs else None
    for i in range(R):
        zt = int(z_t[i])
        if prior == "mask" and zt != V:
            if return_probs:
                probs[i, zt] = 1.0
            continue
        l = logits[i]
        x = np.exp(l - l.max())
        x /= x.sum()
        p = _post.posterior(prior, x, zt, alpha_t, alpha_s)
        if return_probs:
            probs[i] = p
        out[i], gaps[i, 0], gaps[i, 1] = sample_from_probs(prior, p, int(rows[i]), noise)
    return (out, gaps, probs) if return_probs else (out, gaps)


def psi_sample(prior, logits, z_t, alpha_t, alpha_s, kappa, noise, rows=None, return_probs=False):
    """One Psi-sampler step (App. A.4, eq. (psi-sampler)) on a [R, V] logit matrix.

    Same outputs as posterior_sample; every row draws (masked prior: unmasked rows
    choose between keeping their token and the mask)."""
    logits = np.asarray(logits, dtype=np.float64)
    z_t = np.asarray(z_t)
    R, V = logits.shape
    rows = np.arange(R) if rows is None else np.asarray(rows)
    out = np.array(z_t, dtype=np.int64).copy()
    gaps = np.full((R, 2), np.inf)
    K = V + 1 if prior == "mask" else V
    probs = np.zeros((R, K)) if return_probs else None
    for i in range(R):
        zt = int(z_t[i])
        if prior == "mask" and zt != V:
            x = np.zeros(V)
            x[zt] = 1.0
            p = _post.psi_mdm(x, zt, alpha_t, alpha_s, kappa)
        else:
            l = logits[i]
            x = np.exp(l - l.max())
            x /= x.sum()
            p = (_post.psi_mdm if prior == "mask" else _post.psi_usdm)(x, zt, alpha_t, alpha_s, kappa)
        if return_probs:
            probs[i] = p
        out[i], gaps[i, 0], gaps[i, 1] = sample_from_probs(prior, p, int(rows[i]), noise)
    return (out, gaps, probs) if return_probs else (out, gaps)
