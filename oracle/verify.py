"""Speculative verification of a drafted block (test infrastructure only).

Alg. 1 (Psi-Spec, linear sampler) with the standard speculative-decoding
rejection rule it builds on (Sec. 4, one-step diffusion with AR verification):
for one sequence, the verifier gives target distributions p_1..p_B (softmax of
the target logits at the B block positions) and the draft gave proposal
distributions q_1..q_{B-1} and tokens x_1..x_{B-1} (x_i drawn from q_i).  With
uniforms r_i,

  n  = the first i in 1..B-1 with r_i > min(1, p_i(x_i) / q_i(x_i)), else B
  z  ~ Norm([p_n - q_n]_+) if n < B, else z ~ p_B

and the step emits x_1..x_{n-1} followed by z (plus, in Alg. 1, the first
token of the block, which the draft takes from the target model and which is
therefore always accepted).  Every emitted token is distributed as the target
(the rejection correction of speculative decoding), which is what the tests
pin: chi-square of the first emitted token against p_1, and 1 <= TPF =
(n + 1) / 2 <= (B + 1) / 2.

Noise (the definition adopted here, like the posterior draw's): r_i is the word
(STREAM_VERIFY, step, seq, i) read as u = (w + 1/2) 2^-32; z is the two-level
Gumbel-max draw of sampler.py over K = V classes (no mask group) with the level-1
and level-2 words of row `seq`.  Explicit noise: per sequence B - 1 acceptance
words, then the n_top + V words of the draw.  If the residual has no mass (p_n
and q_n equal in every class, which a rejection rules out in exact arithmetic),
z is drawn from p_n.
"""
import numpy as np

from . import philox as _ph
from . import sampler as _sm


def _softmax(l):
    l = np.asarray(l, dtype=np.float64)
    x = np.exp(l - l.max())
    return x / x.sum()


def word_uniform(w):
    return (np.asarray(w, dtype=np.float64) + 0.5) * 2.0 ** -32


class PhiloxVerifyNoise(_sm.PhiloxNoise):
    def accept(self, seq, count):
        return _ph.counter_words(self.seed, _ph.STREAM_VERIFY, self.step, seq, np.arange(count))


class ExplicitVerifyNoise(_sm.ExplicitNoise):
    """Words [S, (B - 1) + n_top + V]: acceptance words first, then the draw's words."""

    def __init__(self, words, B, V):
        words = np.asarray(words, dtype=np.uint32)
        self.acc = words[:, :B - 1]
        super().__init__(words[:, B - 1:], _sm.n_top("uniform", V))

    def accept(self, seq, count):
        return self.acc[seq, :count]


def noise_width(B, V):
    return (B - 1) + _sm.noise_width("uniform", V)


def verify_one(p_logits, q_logits, draft, seq, noise):
    """One sequence: p_logits [B, V], q_logits [B - 1, V], draft [B - 1].

    Returns (n, z, acceptance margins [B - 1] (u - ratio; inf past n), draw gaps (level 1, 2))."""
    p_logits = np.asarray(p_logits, dtype=np.float64)
    B, V = p_logits.shape
    u = word_uniform(noise.accept(seq, B - 1))
    margins = np.full(B - 1, np.inf)
    n = B
    for i in range(B - 1):
        p = _softmax(p_logits[i])
        q = _softmax(q_logits[i])
        x = int(draft[i])
        ratio = min(1.0, p[x] / q[x]) if q[x] > 0 else 1.0
        margins[i] = u[i] - ratio
        if u[i] > ratio:
            n = i + 1
            break
    if n == B:
        dist = _softmax(p_logits[B - 1])
    else:
        resid = np.maximum(_softmax(p_logits[n - 1]) - _softmax(q_logits[n - 1]), 0.0)
        tot = resid.sum()
        dist = resid / tot if tot > 0 else _softmax(p_logits[n - 1])
    z, g1, g2 = _sm.sample_from_probs("uniform", dist, seq, noise)
    return n, z, margins, (g1, g2)


def spec_verify(p_logits, q_logits, draft, noise, seq0=0):
    """S sequences: p_logits [S, B, V], q_logits [S, B - 1, V], draft [S, B - 1].

    Returns n [S], z [S], margins [S, B - 1], gaps [S, 2]."""
    S = p_logits.shape[0]
    out_n = np.zeros(S, dtype=np.int64)
    out_z = np.zeros(S, dtype=np.int64)
    marg = np.zeros((S, p_logits.shape[1] - 1))
    gaps = np.zeros((S, 2))
    for s in range(S):
        out_n[s], out_z[s], marg[s], gaps[s] = verify_one(p_logits[s], q_logits[s], draft[s], seq0 + s, noise)
    return out_n, out_z, marg, gaps
