"""Categorical sampling of z_s from the reverse posterior (test infrastructure only).

The paper draws each token of z_s from its per-position categorical
(App. A.4: the transition is applied token-wise; Sec. 4 linear sampler: each
position is drawn independently) but does not say how a categorical draw is
made.  The reading adopted here is a two-level Gumbel-max draw, exact for any
partition of the classes into groups:

  groups     real classes in contiguous groups of GROUP = 256
             ([0,256), [256,512), ..., [.., V)).
  stage 0    masked prior only: the mask class V is taken iff u < p_V, with
             u = uniform of word (STREAM_TOP, step, row, n_groups) (the word
             after the real groups' level-1 words).  Under App. A.1 eq.
             (mdm-posterior) and App. A.4 eq. (psi-mdm) p_V does not depend on
             x_theta, so this decision needs no logits; otherwise the draw goes
             on over the real classes, whose probabilities sum to 1 - p_V.
  level 1    g* = argmax_g  log M_g + G_g over the real groups,
             M_g = sum_{j in g} p_j, G_g = Gumbel of word (STREAM_TOP, step, row, g).
  level 2    z_s = argmax_{j in g*}  log p_j + G_j,
             G_j = Gumbel of word (STREAM_CLASS, step, row, j).
  ties       the lowest index wins at both levels; log 0 = -inf.

A second reading of level 2 (the "inverse-CDF" draw, used where a group's
candidate must be fixed before the group is known to win, so that one uniform
per group replaces one Gumbel per class):

  level 2'   u_g = uniform of word (STREAM_GROUP_U, step, row, g) for every
             group g; z_s = the first j of g* (in class order) with
             sum_{i in g*, i <= j} p_i > u_{g*} M_{g*}  (if rounding leaves
             none, the last j of g* with p_j > 0).

Level 1 is the same in both readings (same words, same group).  Level 2' picks
j with probability p_j / M_g because u is uniform on (0, 1) and independent of
the level-1 noise, so the pair is again an exact draw from p.

Exactness: stage 0 takes the mask with probability p_V.  The maximum over a
group of log p_j + G_j is distributed as log M_g plus a standard Gumbel and is
independent of the group's argmax, so level 1 picks group g with probability
M_g / sum of the real M's and level 2 picks j with probability p_j / M_g (the
Gumbel-max property; Maddison, Tarlow, Minka, "A* sampling", NeurIPS 2014,
sec. 3).  Together, class j is drawn with probability (1 - p_V) p_j / (1 - p_V).

Explicit-noise layout per row: NU = n_top + V words, the n_top level-1
words first, then one level-2 word per real class.

psi_sample draws from the Psi transition (App. A.4, eq. (psi-sampler), in the
closed forms eqs. (psi-mdm) and (psi-usdm)) with correction strength kappa in
[0, 1]; kappa = 1 is the ancestral step above.  For the masked prior an
unmasked position's x_theta is the one-hot of its token (the carry-over
parameterisation that makes kappa = 1 keep it), so under eq. (psi-mdm) the
token is kept with probability a_s + kappa (1 - a_s) and remasked with
probability (1 - kappa)(1 - a_s) (stage 0 decides); its logits are never read.

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

    def group_u(self, row, g):
        return _ph.counter_words(self.seed, _ph.STREAM_GROUP_U, self.step, row, np.asarray(g))


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


def mask_first(p, row, noise, V):
    """Masked prior, stage 0: the mask class is taken iff u < p_mask, with u the uniform of the
    mask group's level-1 word.  Returns (taken, gap) with gap = |u - p_mask|."""
    u = float(_nz.uniform(noise.top(row, n_top("mask", V))[n_groups_real(V)]))
    pm = float(p[V])
    return u < pm, abs(u - pm)


def sample_from_probs(prior, p, row, noise):
    """Two-level Gumbel-max draw from probabilities p over K classes (masked prior: stage 0
    first, then the two levels over the real classes).

    Returns (class id, level-1 gap, level-2 gap)."""
    V = p.shape[0] - (1 if prior == "mask" else 0)
    bounds = group_bounds("uniform", V)
    gap0 = np.inf
    if prior == "mask":
        taken, gap0 = mask_first(p, row, noise, V)
        if taken:
            return V, gap0, np.inf
    with np.errstate(divide="ignore"):
        logM = np.log(np.array([p[a:b].sum() for a, b in bounds]))
        G = _nz.gumbel(noise.top(row, len(bounds)))
        g, gap1 = _first_argmax_and_gap(logM + G)
        gap1 = min(gap1, gap0)
        a, b = bounds[g]
        idx = np.arange(a, b)
        s = np.log(p[a:b]) + _nz.gumbel(noise.cls(row, idx))
    j, gap2 = _first_argmax_and_gap(s)
    return a + j, gap1, gap2


def inverse_cdf(w, word):
    """Level 2' inside one group: the first index whose running sum of the weights w exceeds
    u * sum(w), u = uniform(word) (the last index with w > 0 if rounding leaves none).

    Returns (index, gap): gap = the distance of u * sum(w) to the nearest running-sum boundary
    that separates two classes of non-zero weight, relative to sum(w) (inf with one such class)."""
    w = np.asarray(w, dtype=np.float64)
    S = w.sum()
    t = float(_nz.uniform(word)) * S
    c = np.cumsum(w)
    above = np.nonzero(c > t)[0]
    pos = np.nonzero(w > 0)[0]
    j = int(above[0]) if above.size else int(pos[-1])
    inner = c[pos[:-1]]                       # boundaries between consecutive classes of mass
    gap = float(np.abs(inner - t).min() / S) if inner.size else np.inf
    return j, gap


def sample_from_probs_cdf(prior, p, row, noise):
    """Two-level draw with the inverse-CDF level 2' (level 1 as sample_from_probs).

    Returns (class id, level-1 gap, level-2 gap); the level-2 gap is relative mass (inverse_cdf)."""
    V = p.shape[0] - (1 if prior == "mask" else 0)
    bounds = group_bounds("uniform", V)
    gap0 = np.inf
    if prior == "mask":
        taken, gap0 = mask_first(p, row, noise, V)
        if taken:
            return V, gap0, np.inf
    with np.errstate(divide="ignore"):
        logM = np.log(np.array([p[a:b].sum() for a, b in bounds]))
        G = _nz.gumbel(noise.top(row, len(bounds)))
    g, gap1 = _first_argmax_and_gap(logM + G)
    gap1 = min(gap1, gap0)
    a, b = bounds[g]
    j, gap2 = inverse_cdf(p[a:b], noise.group_u(row, g))
    return a + j, gap1, gap2


def group_candidates(logits_row, row, noise, V):
    """Level 2' of every real group of one row, each with its own uniform, from logits (the
    within-group distribution of the masked prior's posterior is softmax of the group's logits).
    Returns (candidates [n_groups], gaps [n_groups])."""
    l = np.asarray(logits_row, dtype=np.float64)
    out, gaps = [], []
    for g, (a, b) in enumerate(group_bounds("uniform", V)):
        w = np.exp(l[a:b] - l[a:b].max())
        j, gp = inverse_cdf(w, noise.group_u(row, g))
        out.append(a + j)
        gaps.append(gp)
    return np.array(out), np.array(gaps)


def sample_flat(p, words):
    """Textbook one-Gumbel-per-class draw (used only to pin the two-level draw)."""
    with np.errstate(divide="ignore"):
        return int(np.argmax(np.log(p) + _nz.gumbel(words)))


def posterior_sample(prior, logits, z_t, alpha_t, alpha_s, noise, rows=None, return_probs=False,
                     level2="gumbel"):
    """One reverse step on a [R, V] logit matrix.

    Masked prior: rows whose z_t is not the mask id V are carried over.
    Returns z_s [R] (int64), the per-row level gaps [R, 2] and, optionally,
    the posterior probabilities [R, K].  level2: "gumbel" (level 2) or "cdf" (level 2').
    """
    draw = _draw_fn(level2)
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
        out[i], gaps[i, 0], gaps[i, 1] = draw(prior, p, int(rows[i]), noise)
    return (out, gaps, probs) if return_probs else (out, gaps)


def psi_sample(prior, logits, z_t, alpha_t, alpha_s, kappa, noise, rows=None, return_probs=False,
               level2="gumbel"):
    """One Psi-sampler step (App. A.4, eq. (psi-sampler)) on a [R, V] logit matrix.

    Same outputs as posterior_sample; every row draws (masked prior: unmasked rows
    choose between keeping their token and the mask)."""
    draw = _draw_fn(level2)
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
        out[i], gaps[i, 0], gaps[i, 1] = draw(prior, p, int(rows[i]), noise)
    return (out, gaps, probs) if return_probs else (out, gaps)


def _draw_fn(level2):
    if level2 == "gumbel":
        return sample_from_probs
    if level2 == "cdf":
        return sample_from_probs_cdf
    raise ValueError(f"unknown level-2 rule {level2!r}")
