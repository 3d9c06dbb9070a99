"""GPU parity of parameter init, the posterior/sampling kernel and the Gaussian latent,
through the C ABI, against the float64 oracle on the same seeded inputs."""
import numpy as np
import pytest

import workloads
from oracle import latent as olatent, params as oparams, philox as ophilox, posterior as oposterior, \
    sampler as osampler
from paper_2609_04010_amd import _lib as dd
from tests.gpu_util import (PROB_TOL, compare_ids, dev_i32, dev_words, logits_dev, round_to_dtype,
                            say, torch_or_skip)

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------ parameter initialisation

@pytest.mark.parametrize("c,over", [(1, {}), (2, dict(n_layers=1))])
def test_init_params_matches_oracle(c, over):
    torch = torch_or_skip()
    cfg = workloads.model_cfg(c, **over)
    say("init", c, over)
    seed = workloads.seeds(c)["param"]
    nbytes = dd.param_bytes(cfg)
    buf = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    dd.init_params(cfg, buf, seed=seed)
    host = buf.cpu().numpy()
    specs = oparams.specs(cfg)
    rng = np.random.default_rng(0)
    total = mism = 0
    for tid, (name, shape, _) in enumerate(specs):
        off, r, cc = dd.param_tensor(cfg, tid)
        n = r * cc
        if cfg["dtype"] == "bf16":
            raw = host[off:off + 2 * n].view(np.uint16).astype(np.uint32) << 16
            got = raw.view(np.float32).astype(np.float64)
        else:
            got = host[off:off + 4 * n].view(np.float32).astype(np.float64)
        idx = np.arange(n) if n <= 200_000 else np.sort(rng.choice(n, 200_000, replace=False))
        want = oparams.values_at(cfg, seed, tid, idx)
        diff = got[idx] != want
        total += idx.size
        mism += int(diff.sum())
        if diff.any():   # any disagreement must be a single rounding step of the stored type
            ulp = np.spacing(np.abs(want[diff]).astype(np.float32)).astype(np.float64)
            if cfg["dtype"] == "bf16":
                ulp = ulp * 65536.0
            assert np.all(np.abs(got[idx][diff] - want[diff]) <= ulp * 1.0001), name
    say(f"init: compared {total} elements, {mism} one-ulp differences")
    assert mism <= max(2, total // 1_000_000)


def test_init_params_from_host_blob_roundtrip():
    torch = torch_or_skip()
    cfg = workloads.model_cfg(1, dtype="bf16")
    specs = oparams.specs(cfg)
    P = workloads.host_params(cfg, 11, specs)
    blob = dd.pack_params(cfg, [P[n] for n, _, _ in specs])
    buf = torch.zeros(blob.size, dtype=torch.uint8, device="cuda")
    dd.init_params(cfg, buf, host_blob=blob)
    assert np.array_equal(buf.cpu().numpy(), blob)


# ------------------------------------------------------------------ posterior + sample

POST_CASES = [
    # prior, V, rows, logit dtype, noise, t, s, mask fraction, logit scale, spikes
    ("mask", 32, 128, "fp32", "explicit", 1.0, 0.875, 1.0, 2.0, 0.0),
    ("mask", 32, 128, "fp32", "philox", 0.5, 0.375, 0.5, 2.0, 0.0),
    ("mask", 300, 96, "bf16", "explicit", 0.6, 0.2, 0.7, 3.0, 0.01),
    ("mask", 50257, 40, "bf16", "philox", 1.0, 127 / 128, 1.0, 2.0, 0.0),
    ("mask", 50257, 40, "bf16", "philox", 1 / 128, 0.0, 0.6, 2.0, 0.001),
    ("mask", 50257, 24, "fp32", "philox", 0.5, 0.25, 0.8, 1.0, 0.0),
    ("uniform", 32, 128, "fp32", "explicit", 0.9, 0.8, 0.0, 2.0, 0.0),
    ("uniform", 1000, 64, "bf16", "philox", 0.3, 0.1, 0.0, 3.0, 0.01),
    ("uniform", 50257, 40, "bf16", "philox", 0.75, 0.5, 0.0, 2.0, 0.0),
    ("uniform", 50257, 24, "bf16", "philox", 1 / 64, 0.0, 0.0, 1.0, 0.001),
]


def _run_posterior(torch, prior, V, R, dt, noise, t, s, mf, scale, spikes, seed=5, step=3,
                   want_probs=True, row0=0, kappa=None):
    at, as_ = 1.0 - t, 1.0 - s
    lv = round_to_dtype(workloads.synthetic_logits(seed, R, V, scale=scale, spike_frac=spikes), dt)
    if prior == "mask":
        zt = workloads.masked_state(seed + 1, 1, R, V, mf).reshape(-1)
    else:
        zt = workloads.uniform_state(seed + 1, 1, R, V).reshape(-1)
    ld = int(dd.logits_ld(V))
    lg = logits_dev(torch, lv, dt, ld)
    zt_d = dev_i32(torch, zt)
    zs_d = torch.empty_like(zt_d)
    K = V + 1 if prior == "mask" else V
    probs = torch.zeros((R, K), dtype=torch.float32, device="cuda") if want_probs else None
    rlse = torch.full((R,), float("nan"), dtype=torch.float32, device="cuda")
    ntop = osampler.n_top(prior, V)
    if noise == "explicit":
        words = workloads.noise_words(seed + 2, (R, osampler.noise_width(prior, V)))
        nz = osampler.ExplicitNoise(words, ntop)
        wd = dev_words(torch, words)
    else:
        nz = osampler.PhiloxNoise(seed + 3, step)
        wd = None
    rows = np.arange(R) + row0
    if kappa is None:
        dd.posterior_sample(prior, lg, dt, ld, R, V, zt_d, at, as_, zs_d, noise_words=wd, seed=seed + 3,
                            step=step, row0=row0, probs=probs, row_lse=rlse)
        ref, gaps, rprobs = osampler.posterior_sample(prior, lv, zt, at, as_, nz, rows=rows,
                                                      return_probs=True)
    else:
        dd.psi_posterior_sample(prior, lg, dt, ld, R, V, zt_d, at, as_, kappa, zs_d, noise_words=wd,
                                seed=seed + 3, step=step, row0=row0, probs=probs, row_lse=rlse)
        ref, gaps, rprobs = osampler.psi_sample(prior, lv, zt, at, as_, kappa, nz, rows=rows,
                                                return_probs=True)
    _last_row_lse[:] = [lv, rlse.cpu().numpy()]
    return zt, zs_d.cpu().numpy(), ref, gaps, rprobs, (probs.cpu().numpy() if want_probs else None)


_last_row_lse = [None, None]   # (logits, row_lse output) of the latest _run_posterior call


@pytest.mark.parametrize("case", POST_CASES, ids=lambda c: f"{c[0]}-V{c[1]}-{c[3]}-{c[4]}-t{c[5]:.3f}")
def test_posterior_parity(case):
    torch = torch_or_skip()
    say("posterior", case)
    prior, V = case[0], case[1]
    zt, got, ref, gaps, rprobs, gprobs = _run_posterior(torch, *case)
    compare_ids(got, ref, gaps, f"posterior {prior} V={V}")
    perr = float(np.abs(gprobs - rprobs).max())
    say(f"max |dp| = {perr:.3e}")
    assert perr <= PROB_TOL
    # the draw's own fp32 row log-sum-exp: drawn rows get it, carried-over rows are left untouched;
    # the probabilities it implies meet the same bar
    lv, rl = _last_row_lse
    drawn = (zt == V) if prior == "mask" else np.ones(zt.size, bool)
    assert np.isnan(rl[~drawn]).all() and np.isfinite(rl[drawn]).all()
    m = lv.max(axis=1)
    lse = m + np.log(np.exp(lv - m[:, None]).sum(axis=1))
    at, as_ = 1.0 - case[5], 1.0 - case[6]
    dpl = 0.0
    for r in np.nonzero(drawn)[0]:
        p = oposterior.posterior(prior, np.exp(lv[r] - float(rl[r])), int(zt[r]), at, as_)
        dpl = max(dpl, float(np.abs(p - rprobs[r]).max()))
    say(f"row lse: max |d| = {np.abs(rl[drawn] - lse[drawn]).max():.3e}; implied max |dp| = {dpl:.3e}")
    assert dpl <= PROB_TOL
    if prior == "mask":
        keep = zt != V
        assert np.array_equal(got[keep], zt[keep])          # carry-over, bit exact
        assert np.all(got[~keep] <= V)
    assert np.all((got >= 0) & (got < (V + 1 if prior == "mask" else V)))


PSI_CASES = [
    # prior, V, rows, logit dtype, noise, t, s, mask fraction, logit scale, spikes, kappa
    ("mask", 32, 256, "fp32", "explicit", 0.5, 0.375, 0.5, 2.0, 0.0, 0.0),
    ("mask", 300, 256, "bf16", "philox", 0.6, 0.4, 0.5, 3.0, 0.01, 0.5),
    ("mask", 50257, 48, "bf16", "philox", 0.75, 0.5, 0.6, 2.0, 0.0, 0.3),
    ("uniform", 32, 128, "fp32", "explicit", 0.9, 0.8, 0.0, 2.0, 0.0, 0.0),
    ("uniform", 1000, 64, "bf16", "philox", 0.3, 0.1, 0.0, 3.0, 0.01, 0.6),
    ("uniform", 50257, 32, "bf16", "philox", 0.75, 0.5, 0.0, 2.0, 0.0, 0.25),
]


@pytest.mark.parametrize("case", PSI_CASES, ids=lambda c: f"{c[0]}-V{c[1]}-{c[3]}-{c[4]}-k{c[10]}")
def test_psi_posterior_parity(case):
    """App. A.4 Psi transition with kappa < 1 against the oracle on the same (device-rounded)
    logits and noise; masked prior: unmasked rows keep their token or become the mask."""
    torch = torch_or_skip()
    say("psi posterior", case)
    prior, V, kappa = case[0], case[1], case[10]
    zt, got, ref, gaps, rprobs, gprobs = _run_posterior(torch, *case[:10], kappa=kappa)
    compare_ids(got, ref, gaps, f"psi {prior} V={V} kappa={kappa}")
    perr = float(np.abs(gprobs - rprobs).max())
    say(f"max |dp| = {perr:.3e}")
    assert perr <= PROB_TOL
    if prior == "mask":
        dec = zt != V
        assert np.all((got[dec] == zt[dec]) | (got[dec] == V))
        assert np.any(got[dec] == V)                       # some decoded tokens were remasked
    assert np.all((got >= 0) & (got < (V + 1 if prior == "mask" else V)))


def test_psi_at_kappa_one_equals_the_posterior_entry_point():
    torch = torch_or_skip()
    for case in (POST_CASES[2], POST_CASES[3], POST_CASES[8]):
        say("psi kappa=1", case)
        _, a, _, _, _, pa = _run_posterior(torch, *case)
        _, b, _, _, _, pb = _run_posterior(torch, *case, kappa=1.0)
        assert np.array_equal(a, b) and np.array_equal(pa, pb)


def test_psi_explicit_words_equal_in_kernel_philox_and_unmasked_logits_unread():
    torch = torch_or_skip()
    V, R = 600, 96
    lv = round_to_dtype(workloads.synthetic_logits(3, R, V, scale=0.5), "bf16")
    zt = workloads.masked_state(4, 1, R, V, 0.5).reshape(-1)
    ld = int(dd.logits_ld(V))
    lg = logits_dev(torch, lv, "bf16", ld)
    poisoned = lv.copy()
    poisoned[zt != V] = np.nan
    lp = logits_dev(torch, poisoned, "bf16", ld)
    rows = np.arange(R)[:, None]
    ntop = osampler.n_top("mask", V)
    words = np.concatenate([ophilox.counter_words(5, ophilox.STREAM_TOP, 2, rows, np.arange(ntop)[None]),
                            ophilox.counter_words(5, ophilox.STREAM_CLASS, 2, rows, np.arange(V)[None])], 1)
    zd = dev_i32(torch, zt)
    outs = []
    for logits, wd in ((lg, None), (lg, dev_words(torch, words)), (lp, None)):
        o = torch.empty(R, dtype=torch.int32, device="cuda")
        dd.psi_posterior_sample("mask", logits, "bf16", ld, R, V, zd, 0.4, 0.6, 0.2, o, noise_words=wd,
                                seed=5, step=2)
        outs.append(o.cpu().numpy())
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_posterior_row_offset_keys_noise_by_global_row():
    torch = torch_or_skip()
    case = ("mask", 300, 64, "bf16", "philox", 0.6, 0.3, 1.0, 3.0, 0.0)
    _, got, ref, gaps, _, _ = _run_posterior(torch, *case, row0=1000, want_probs=False)
    compare_ids(got, ref, gaps, "posterior row0=1000")


def test_explicit_words_equal_in_kernel_philox():
    """The device Philox must produce exactly the oracle's words: feeding the oracle's words as
    explicit noise gives the same draw as the in-kernel generator."""
    torch = torch_or_skip()
    for prior, V, R in (("mask", 600, 64), ("uniform", 50257, 16)):
        say("explicit==philox", prior, V)
        lv = round_to_dtype(workloads.synthetic_logits(1, R, V, scale=0.5), "bf16")
        zt = (workloads.all_mask(1, R, V) if prior == "mask" else workloads.uniform_state(2, 1, R, V)).reshape(-1)
        ld = int(dd.logits_ld(V))
        lg = logits_dev(torch, lv, "bf16", ld)
        rows = np.arange(R)[:, None]
        ntop = osampler.n_top(prior, V)
        words = np.concatenate([ophilox.counter_words(77, ophilox.STREAM_TOP, 9, rows, np.arange(ntop)[None]),
                                ophilox.counter_words(77, ophilox.STREAM_CLASS, 9, rows, np.arange(V)[None])], 1)
        a = torch.empty(R, dtype=torch.int32, device="cuda")
        b = torch.empty_like(a)
        zd = dev_i32(torch, zt)
        dd.posterior_sample(prior, lg, "bf16", ld, R, V, zd, 0.4, 0.6, a, seed=77, step=9)
        dd.posterior_sample(prior, lg, "bf16", ld, R, V, zd, 0.4, 0.6, b, noise_words=dev_words(torch, words))
        assert torch.equal(a, b)


def test_posterior_in_place_and_deterministic():
    torch = torch_or_skip()
    V, R = 50257, 64
    lv = round_to_dtype(workloads.synthetic_logits(4, R, V), "bf16")
    zt = workloads.masked_state(5, 1, R, V, 0.5).reshape(-1)
    ld = int(dd.logits_ld(V))
    lg = logits_dev(torch, lv, "bf16", ld)
    out = torch.empty(R, dtype=torch.int32, device="cuda")
    dd.posterior_sample("mask", lg, "bf16", ld, R, V, dev_i32(torch, zt), 0.3, 0.5, out, seed=1, step=2)
    z = dev_i32(torch, zt)
    dd.posterior_sample("mask", lg, "bf16", ld, R, V, z, 0.3, 0.5, z, seed=1, step=2)   # z_s aliases z_t
    assert torch.equal(out, z)


def test_poisoned_carry_over_rows_are_never_read():
    torch = torch_or_skip()
    V, R = 50257, 32
    lv = round_to_dtype(workloads.synthetic_logits(6, R, V), "bf16")
    zt = workloads.masked_state(7, 1, R, V, 0.5).reshape(-1)
    lv[zt != V] = np.nan
    ld = int(dd.logits_ld(V))
    lg = logits_dev(torch, lv, "bf16", ld)
    out = torch.empty(R, dtype=torch.int32, device="cuda")
    dd.posterior_sample("mask", lg, "bf16", ld, R, V, dev_i32(torch, zt), 0.3, 0.5, out, seed=1, step=2)
    got = out.cpu().numpy()
    ref, gaps = osampler.posterior_sample("mask", np.nan_to_num(lv), zt, 0.3, 0.5, osampler.PhiloxNoise(1, 2))
    compare_ids(got, ref, gaps, "poisoned")


def test_out_of_range_tokens_set_the_device_error_word():
    torch = torch_or_skip()
    V, R = 64, 8
    lv = round_to_dtype(workloads.synthetic_logits(8, R, V), "fp32")
    ld = int(dd.logits_ld(V))
    lg = logits_dev(torch, lv, "fp32", ld)
    zt = np.full(R, V, dtype=np.int32)
    zt[3] = V + 7
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = torch.empty(R, dtype=torch.int32, device="cuda")
    dd.posterior_sample("mask", lg, "fp32", ld, R, V, dev_i32(torch, zt), 0.3, 0.5, out, seed=1,
                        step=2, dev_err=err)
    assert dd.read_device_error(err) == dd.DD_DEVERR_TOKEN
    assert np.all(out.cpu().numpy() <= V)


# ------------------------------------------------------------------ Gaussian latent

@pytest.mark.parametrize("V,R,at", [(7, 512, 0.0), (7, 512, 0.6), (50257, 48, 0.0), (50257, 48, 0.9),
                                    (50257, 48, 0.999)])
def test_gaussian_latent_parity(V, R, at):
    torch = torch_or_skip()
    say("latent", V, R, at)
    sigma = float(np.sqrt(1 - at * at))
    x = workloads.clean_tokens(12, 1, R, V).reshape(-1)
    z = torch.empty(R, dtype=torch.int32, device="cuda")
    dd.gaussian_latent_argmax(dev_i32(torch, x), R, V, at, sigma, seed=321, step=4, z_out=z)
    ref = olatent.latent_argmax(x, V, at, sigma, seed=321, step=4)
    got = z.cpu().numpy()
    say(f"latent agree={np.mean(got == ref):.6f} kept={np.mean(ref == x):.4f}")
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("prior,dt", [("mask", "bf16"), ("uniform", "bf16"), ("mask", "fp32"), ("uniform", "fp32")])
def test_degenerate_logit_rows_are_reported_and_keep_their_token(prior, dt):
    """Rows with NaN, +inf or (uniform prior) no finite logit: DD_DEVERR_LOGITS, z_s = z_t there,
    every other row bit-identical to the same call without those rows."""
    torch = torch_or_skip()
    say("degenerate rows", prior, dt)
    R, V = 64, 700
    lv = round_to_dtype(workloads.synthetic_logits(21, R, V, scale=2.0), dt)
    zt = (np.full(R, V) if prior == "mask" else workloads.uniform_state(22, 1, R, V).reshape(-1)).astype(np.int64)
    bad = {3: np.nan, 17: np.inf, 40: "allneg"}
    lb = lv.copy()
    for r, v in bad.items():
        if v == "allneg":
            lb[r, :] = -np.inf
        else:
            lb[r, 123] = v
    ld = int(dd.logits_ld(V))
    outs = []
    for vals in (lv, lb):
        lg = logits_dev(torch, vals, dt, ld)
        zt_d = dev_i32(torch, zt)
        zs_d = torch.empty_like(zt_d)
        err = torch.zeros(1, dtype=torch.int32, device="cuda")
        dd.posterior_sample(prior, lg, dt, ld, R, V, zt_d, 0.3, 0.6, zs_d, seed=9, step=4, dev_err=err)
        outs.append((zs_d.cpu().numpy(), dd.read_device_error(err)))
    (clean, e0), (dirty, e1) = outs
    assert e0 == 0
    flagged = list(bad)
    assert e1 == dd.DD_DEVERR_LOGITS
    for r in range(R):
        if r in flagged:
            assert dirty[r] == zt[r], (r, dirty[r])
        else:
            assert dirty[r] == clean[r], r
    assert ((dirty >= 0) & (dirty <= V)).all()
