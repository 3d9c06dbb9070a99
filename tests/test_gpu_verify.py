"""GPU parity of the speculative verification (dd_spec_verify) against the oracle (Alg. 1)."""
import numpy as np
import pytest

import workloads
from oracle import philox as ophilox, sampler as osampler, verify as overify
from paper_2609_04010_amd import _lib as dd
from tests.gpu_util import (GAP, compare_ids, dev_i32, dev_words, logits_dev, round_to_dtype, say,
                            torch_or_skip)

pytestmark = pytest.mark.gpu

ACC_MARGIN = 1e-4   # acceptance decisions must agree wherever |u - min(1, p/q)| exceeds this


def _softmax(l):
    x = np.exp(l - l.max(-1, keepdims=True))
    return x / x.sum(-1, keepdims=True)


def _case(seed, S, B, V, dt, closeness, scale=2.0):
    """Target / draft logits (draft = target + noise of the given size) and drafts drawn from q."""
    r = np.random.default_rng(seed)
    pl = round_to_dtype(workloads.synthetic_logits(seed, S * B, V, scale=scale), dt).reshape(S, B, V)
    ql = round_to_dtype(pl[:, :-1].reshape(-1, V) + closeness * r.standard_normal((S * (B - 1), V)), dt)
    ql = ql.reshape(S, B - 1, V)
    q = _softmax(ql)
    draft = np.array([[r.choice(V, p=q[s, i]) for i in range(B - 1)] for s in range(S)], dtype=np.int64)
    return pl, ql, draft


def _run_gpu(torch, pl, ql, draft, dt, words=None, seed=0, step=0, row0=0):
    S, B, V = pl.shape
    ld = int(dd.logits_ld(V))
    p_d = logits_dev(torch, pl.reshape(S * B, V), dt, ld)
    q_d = logits_dev(torch, ql.reshape(S * (B - 1), V), dt, ld) if B > 1 else None
    n = torch.empty(S, dtype=torch.int32, device="cuda")
    z = torch.empty_like(n)
    ws = torch.zeros(dd.spec_verify_workspace_bytes(S, B), dtype=torch.uint8, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    dd.spec_verify(p_d, q_d, dt, ld, S, B, V, dev_i32(torch, draft) if B > 1 else None, n, z, ws,
                   noise_words=dev_words(torch, words) if words is not None else None, seed=seed, step=step,
                   row0=row0, dev_err=err)
    assert int(err.item()) == 0
    return n.cpu().numpy(), z.cpu().numpy()


CASES = [
    # S, B, V, dtype, noise, closeness of draft to target
    (256, 4, 32, "fp32", "explicit", 0.5),
    (128, 8, 600, "bf16", "philox", 0.3),
    (64, 16, 50257, "bf16", "philox", 0.2),
    (48, 5, 50257, "fp32", "explicit", 1.0),
    (64, 1, 1000, "bf16", "philox", 0.0),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"S{c[0]}-B{c[1]}-V{c[2]}-{c[3]}-{c[4]}")
def test_spec_verify_parity(case):
    torch = torch_or_skip()
    S, B, V, dt, noise, close = case
    say("spec_verify", case)
    pl, ql, draft = _case(7, S, B, V, dt, close) if B > 1 else (
        round_to_dtype(workloads.synthetic_logits(7, S, V), dt).reshape(S, 1, V), np.zeros((S, 0, V)),
        np.zeros((S, 0), dtype=np.int64))
    if noise == "explicit":
        words = workloads.noise_words(11, (S, overify.noise_width(B, V)))
        nz = overify.ExplicitVerifyNoise(words, B, V)
        n, z = _run_gpu(torch, pl, ql, draft, dt, words=words)
    else:
        nz = overify.PhiloxVerifyNoise(13, 6)
        n, z = _run_gpu(torch, pl, ql, draft, dt, seed=13, step=6, row0=0)
    rn, rz, marg, gaps = overify.spec_verify(pl, ql, draft, nz)
    # acceptance: exact where every tested margin up to the oracle's n is clear
    clear = np.array([np.all(np.abs(marg[s][:min(rn[s], B - 1)]) > ACC_MARGIN) for s in range(S)])
    bad = np.nonzero(clear & (n != rn))[0]
    say(f"n: agree {np.mean(n == rn):.4f}, clear {clear.sum()}, clear mismatches {bad.size}; "
        f"mean n {n.mean():.2f}")
    assert bad.size == 0 and np.mean(n == rn) >= 0.99
    same = n == rn
    compare_ids(z[same], rz[same], gaps[same], f"spec_verify z {case}")
    tpf = (n + 1) / 2
    assert tpf.min() >= 1 and tpf.max() <= (B + 1) / 2


def test_spec_verify_explicit_words_equal_philox():
    torch = torch_or_skip()
    S, B, V = 32, 6, 700
    pl, ql, draft = _case(3, S, B, V, "bf16", 0.4)
    seqs = np.arange(S)[:, None] + 100
    ntop = osampler.n_top("uniform", V)
    words = np.concatenate([ophilox.counter_words(21, ophilox.STREAM_VERIFY, 2, seqs, np.arange(B - 1)[None]),
                            ophilox.counter_words(21, ophilox.STREAM_TOP, 2, seqs, np.arange(ntop)[None]),
                            ophilox.counter_words(21, ophilox.STREAM_CLASS, 2, seqs, np.arange(V)[None])], 1)
    a = _run_gpu(torch, pl, ql, draft, "bf16", seed=21, step=2, row0=100)
    b = _run_gpu(torch, pl, ql, draft, "bf16", words=words)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_spec_verify_identical_draft_accepts_the_block():
    torch = torch_or_skip()
    S, B, V = 40, 8, 900
    pl, _, _ = _case(5, S, B, V, "bf16", 0.0)
    draft = np.random.default_rng(2).integers(0, V, (S, B - 1))
    n, _ = _run_gpu(torch, pl, pl[:, :-1].copy(), draft, "bf16", seed=1, step=1)
    assert np.all(n == B)


def test_spec_verify_is_lossless_chi2():
    """The first emitted token (x_1 if accepted, else the replacement) follows p_1 on the GPU too."""
    torch = torch_or_skip()
    from scipy import stats
    V, B, S = 12, 2, 40000
    r = np.random.default_rng(4)
    p1 = round_to_dtype(1.5 * r.standard_normal(V), "fp32")
    q1 = round_to_dtype(1.5 * r.standard_normal(V) + np.linspace(0, 2, V), "fp32")
    pl = np.broadcast_to(np.stack([p1, p1]), (S, B, V)).copy()
    ql = np.broadcast_to(q1, (S, B - 1, V)).copy()
    draft = r.choice(V, size=(S, 1), p=_softmax(q1))
    n, z = _run_gpu(torch, pl, ql, draft, "fp32", seed=8, step=3)
    first = np.where(n > 1, draft[:, 0], z)
    counts = np.bincount(first, minlength=V).astype(float)
    pvalue = stats.chisquare(counts, _softmax(p1) * S).pvalue
    say(f"lossless chi2 p = {pvalue:.4f}; acceptance {np.mean(n > 1):.3f}")
    assert pvalue > 1e-3


def test_spec_verify_degenerate_logits_are_reported():
    """NaN in every target row of one sequence, a NaN inside an otherwise -inf 16-byte chunk of every
    target row of another (the thread reading that chunk meets no finite logit), +inf in every
    target row of a third: DD_DEVERR_LOGITS and z = 0 there.  NaN in the draft rows of another: its
    draw stays valid (the residual falls back to p).  Every other sequence is bit-identical to the
    clean call."""
    torch = torch_or_skip()
    S, B, V, dt = 8, 4, 600, "bf16"
    pl, ql, draft = _case(17, S, B, V, dt, 0.3)
    pd, qd = pl.copy(), ql.copy()
    pd[2, :, 5] = np.nan
    pd[3, :, 16:24] = -np.inf
    pd[3, :, 21] = np.nan
    pd[6, :, 9] = np.inf
    qd[5, :, 7] = np.nan
    ld = int(dd.logits_ld(V))
    res = []
    for p_, q_ in ((pl, ql), (pd, qd)):
        p_d = logits_dev(torch, p_.reshape(S * B, V), dt, ld)
        q_d = logits_dev(torch, q_.reshape(S * (B - 1), V), dt, ld)
        n = torch.empty(S, dtype=torch.int32, device="cuda")
        z = torch.empty_like(n)
        ws = torch.zeros(dd.spec_verify_workspace_bytes(S, B), dtype=torch.uint8, device="cuda")
        err = torch.zeros(1, dtype=torch.int32, device="cuda")
        dd.spec_verify(p_d, q_d, dt, ld, S, B, V, dev_i32(torch, draft), n, z, ws, seed=3, step=1, dev_err=err)
        res.append((n.cpu().numpy(), z.cpu().numpy(), dd.read_device_error(err)))
    (n0, z0, e0), (n1, z1, e1) = res
    say(f"clean err {e0}, dirty err {e1}; seq 2 -> ({n1[2]}, {z1[2]}), seq 5 -> ({n1[5]}, {z1[5]})")
    assert e0 == 0 and e1 == dd.DD_DEVERR_LOGITS
    assert z1[2] == 0 and z1[3] == 0 and z1[6] == 0 and 1 <= n1[5] <= B and 0 <= z1[5] < V
    keep = [s for s in range(S) if s not in (2, 3, 5, 6)]
    assert np.array_equal(n0[keep], n1[keep]) and np.array_equal(z0[keep], z1[keep])
